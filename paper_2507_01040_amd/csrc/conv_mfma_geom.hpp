// Address arithmetic of conv_mfma_kernel (k = 2, 3): which input rows and
// filters a workgroup stages, where each lane's direct global->LDS loads read
// and land, which LDS words each MFMA fragment reads, and where each output
// goes.  The kernel and the host-side bounds checker (a CPU build of the
// library used by the tests) both call these functions, so the checker
// verifies the kernel's own arithmetic.
#pragma once

#include <stdint.h>

#include "common.hpp"

namespace cliff {

struct MfmaArgs {
    const float* x;
    const float* w;
    const float* bias;
    float* y;
    int C_in, C_out, D, Do, df;
    int M;          // number of output positions B * d_out^k
    int npos;       // d_out^k
    int cc;         // input channels per stage
    int n_stage;    // ceil(C_in / cc) (k = 2) or that times d_filter (k = 3)
    int n_co_blk, n_blk;
    int rowblk;     // 2D row-aligned blocks with column-window slabs (wide images)
    int nseg;       // row-aligned blocks: blocks per output row
    int sw;         // row-aligned blocks: slab row width in positions
    int stage_floats;  // LDS floats of one stage buffer
    SignMasks sign;
    ActParams act;
};

// The compile-time shape of one kernel instantiation, as plain ints: KD
// spatial dimensions, NB blades, DF filter size (0: run time), CCT channels
// per stage (0: run time), WCO x WPOS waves of MW x NW MFMA tiles (16 x 16),
// SLOTS staging slots per lane, the K loop split over WK waves.  NEG: LDS
// also holds the filters negated (loaded again through registers and written
// negated), and each A lane reads the copy of its table sign instead of
// multiplying by it (one channel per stage, no zero sign).
struct MfmaTile {
    int KD, NB, DF, CCT, WCO, WPOS, MW, NW, SLOTS, WK, NEG;
    __host__ __device__ constexpr int nt() const { return 64 * WCO * WPOS * WK; }
    __host__ __device__ constexpr int cpt() const { return 16 / NB; }  // channels per tile
    __host__ __device__ constexpr int co_wg() const { return WCO * MW * (16 / NB); }
    __host__ __device__ constexpr int pos() const { return WPOS * NW * 16; }
    __host__ __device__ constexpr int nh() const { return NB / 4; }  // 4-blade groups
    // NEG: float4 of filters per lane and stage (registers of the negated copy)
    __host__ __device__ constexpr int fslots() const
    {
        return NEG ? (co_wg() * DF * DF * NB / 4 + nt() - 1) / nt() : 0;
    }
};

// Quotient of non-negative ints, as an unsigned division (a shorter
// instruction sequence than the signed one); every index divided here is
// non-negative.
__host__ __device__ inline int udiv(int a, int b) { return (int)((unsigned)a / (unsigned)b); }

// Division of non-negative ints below 2^31 by a divisor fixed for the block,
// through its reciprocal m = ceil(2^32 / d), formed once: the high word of
// n m exceeds n / d by less than n / 2^32 < 1/2, so it is the quotient or one
// more, and the sign of the remainder decides (d = 1, whose m needs 33 bits,
// is taken apart).  Per division a multiply-high, a multiply and a compare
// instead of a full division sequence.
struct FastDiv {
    int d;
    unsigned m;
};
__host__ __device__ inline FastDiv fast_div(int d)
{
    return FastDiv{d, d > 1 ? 0xFFFFFFFFu / (unsigned)d + 1u : 0u};
}
__host__ __device__ inline int fdiv(int n, const FastDiv& f)
{
    if (f.d == 1) return n;
    const unsigned q = (unsigned)(((unsigned long long)(unsigned)n * f.m) >> 32);
    // q d <= n + d < 2^32: the product does not wrap in 32 unsigned bits
    return (int)(q * (unsigned)f.d > (unsigned)n ? q - 1 : q);
}

// Geometry of one workgroup's block: P consecutive flattened output positions
// [m0, m_end) (or, with row-aligned blocks, at most P positions of one output
// row starting at column x0) by CO_WG output channels from co0, and the slab
// of input rows it stages per channel.
struct MfmaBlock {
    int co0, m0, m_end, x0;
    int pl0, ylo0, len0, n_rows;  // slab: first plane, its first row, rows in it, total rows
    int b0, z0;                   // batch entry (and, for k = 3, plane) of the first row
    int df, taps2, taps_full, D, Do;
    int row_floats, lrow_floats;  // global and LDS row strides
    int cc, slab_f4, wq_f4, wch_f4, total_f4, w_lds, w_neg;
    int plane_floats, x_cstride, w_cstride;
    FastDiv fslab, flrow, fD, fDo;  // the per-lane divisors, as reciprocals
    bool rb;
};

__host__ __device__ inline MfmaBlock mfma_block(const MfmaTile& T, const MfmaArgs& a, int bid)
{
    MfmaBlock g;
    g.df = T.DF > 0 ? T.DF : a.df;
    g.taps2 = g.df * g.df;
    g.taps_full = T.KD == 2 ? g.taps2 : g.taps2 * g.df;
    g.D = a.D;
    g.Do = a.Do;
    const int D = g.D, Do = g.Do, NB = T.NB, P = T.pos();
    g.row_floats = D * NB;
    g.rb = T.KD == 2 && a.rowblk;
    g.lrow_floats = g.rb ? a.sw * NB : g.row_floats;

    // Workgroups are dispatched round-robin over the 8 XCDs; renumbered so
    // each XCD (own L2) works through a contiguous run of position blocks,
    // whose input slabs overlap.
    const int per = a.n_blk >> 3, rem = a.n_blk & 7;
    const int xcd = bid & 7, slot = bid >> 3;
    const int tile = xcd < rem ? xcd * (per + 1) + slot
                               : rem * (per + 1) + (xcd - rem) * per + slot;
    const int pos_blk = udiv(tile, a.n_co_blk);
    const int co_blk = tile - pos_blk * a.n_co_blk;
    g.co0 = co_blk * T.co_wg();
    g.x0 = 0;
    if (g.rb) {
        const int ry = udiv(pos_blk, a.nseg), seg = pos_blk - ry * a.nseg;  // output row over (b, y)
        g.x0 = seg * P;
        g.m0 = ry * Do + g.x0;
        g.m_end = g.m0 + (P < Do - g.x0 ? P : Do - g.x0);
    } else {
        g.m0 = pos_blk * P;
        g.m_end = g.m0 + P < a.M ? g.m0 + P : a.M;
    }

    // Output rows r0..r1 (rows of d_out positions), planes pl0..pl1 (2D:
    // batch entry; 3D: (batch, z)).  Each plane contributes its output rows
    // plus d_filter - 1 halo rows; full middle planes all d_image rows.
    const int r0 = udiv(g.m0, Do), r1 = udiv(g.m_end - 1, Do);
    g.pl0 = udiv(r0, Do);
    const int pl1 = udiv(r1, Do);
    g.ylo0 = r0 - g.pl0 * Do;
    g.len0 = g.pl0 == pl1 ? (r1 - r0) + g.df : D - g.ylo0;
    g.n_rows = g.pl0 == pl1 ? g.len0
                            : g.len0 + (pl1 - g.pl0 - 1) * D + (r1 - pl1 * Do) + g.df;

    g.cc = T.CCT > 0 ? T.CCT : a.cc;
    g.slab_f4 = g.n_rows * (g.lrow_floats / 4);  // one channel's slab
    g.wq_f4 = g.taps2 * NB / 4;
    g.wch_f4 = T.co_wg() * g.wq_f4;              // one channel's filters
    // float4 staged by direct loads
    g.total_f4 = g.cc * (g.slab_f4 + g.wch_f4);
    g.w_lds = g.cc * g.slab_f4 * 4;              // float offset of the filters in a buffer
    g.w_neg = g.w_lds + g.cc * g.wch_f4 * 4;     // NEG: of their negated copy
    g.b0 = T.KD == 2 ? g.pl0 : udiv(g.pl0, Do);
    g.z0 = T.KD == 2 ? 0 : g.pl0 - g.b0 * Do;
    g.plane_floats = D * g.row_floats;           // one d_image x d_image plane
    g.x_cstride = g.plane_floats * (T.KD == 3 ? D : 1);  // < 2^31 (host check)
    g.w_cstride = a.C_out * g.taps_full * NB;
    g.fslab = fast_div(g.slab_f4);
    g.flrow = fast_div(g.lrow_floats / 4);
    g.fD = fast_div(D);
    g.fDo = fast_div(Do);
    return g;
}

// Float offset, from the stage's filter base, of float4 e of the stage's
// filters [cc][co][tap][blade] in LDS order (channels past C_out read the
// last channel; their results are never stored).
__host__ __device__ inline int mfma_filter_src(const MfmaTile& T, const MfmaArgs& a,
                                               const MfmaBlock& g, int e)
{
    const int c_l = udiv(e, g.wch_f4);
    const int e2 = e - c_l * g.wch_f4;
    const int co_l = udiv(e2, g.wq_f4);
    const int r4 = e2 - co_l * g.wq_f4;
    const int co = g.co0 + co_l < a.C_out - 1 ? g.co0 + co_l : a.C_out - 1;
    return c_l * g.w_cstride + (co - g.co0) * g.taps_full * T.NB + r4 * 4;
}

// NEG: filter register slot u of lane tid holds float4 e = u * NT + tid of
// the stage's filters (when e < cc * wch_f4); it is written to LDS negated at
// mfma_wreg_lds(g, e, 1) (mfma_wreg_lds(g, e, 0) is where the direct loads
// put it as it is).
__host__ __device__ inline int mfma_wreg_lds(const MfmaBlock& g, int e, int neg)
{
    return (neg ? g.w_neg : g.w_lds) + 4 * e;
}

// Staging.  A stage buffer holds float4 slots in staging order: cc channel
// slabs [cc][slab rows] in [0, cc * slab_f4), then cc channels of filters
// [cc][co][tap][blade] (NEG: then their negated copy, which does not go
// through the direct-load slots but through registers, mfma_wreg_*).  Float4 f = t * NT + tid of the buffer is slot t of
// lane tid.  Returns its source offset: >= 0, the input float offset from the
// stage's slab base; < 0, -1 - the filter float offset from the stage's filter
// base (channels past C_out read the last channel; their results are never
// stored).  N_B = 8 rows are stored [half][x][4] (slot sr = half * D + x holds
// the global float4 2 x + half of the row); row-aligned blocks stage columns
// x0 .. x0 + sw - 1.
__host__ __device__ inline int mfma_slot_goff(const MfmaTile& T, const MfmaArgs& a,
                                              const MfmaBlock& g, int f)
{
    const int NB = T.NB, D = g.D, Do = g.Do;
    const int lrow_f4 = g.lrow_floats / 4;
    if (f < g.cc * g.slab_f4) {
        const int c_l = fdiv(f, g.fslab);
        const int fr = f - c_l * g.slab_f4;
        const int row = fdiv(fr, g.flrow);
        const int sr = fr - row * lrow_f4;
        const int colr = g.x0 + sr < D - 1 ? g.x0 + sr : D - 1;
        const int col = NB == 8 ? 2 * (sr - fdiv(sr, g.fD) * D) + fdiv(sr, g.fD) : (g.rb ? colr : sr);
        int pl, yin;
        if (row < g.len0) {
            pl = g.pl0;
            yin = g.ylo0 + row;
        } else {
            const int s2 = row - g.len0;
            pl = g.pl0 + 1 + fdiv(s2, g.fD);
            yin = s2 - fdiv(s2, g.fD) * D;
        }
        int rel;  // planes between pl0's first row and this row's plane
        if (T.KD == 2) {
            rel = (pl - g.pl0) * a.C_in;
        } else {
            const int b = fdiv(pl, g.fDo), z = pl - b * Do;
            rel = ((b - g.b0) * a.C_in * D + (z - g.z0));
        }
        return c_l * g.x_cstride + rel * g.plane_floats + yin * g.row_floats + col * 4;
    }
    if (f < g.total_f4) return -1 - mfma_filter_src(T, a, g, f - g.cc * g.slab_f4);
    return 0;
}

// Whether slot float4 f (source offset goff) is loaded in a stage with nv
// valid channels.  Slots are channel-major within each section, so a stage
// with nv < cc valid channels loads f < nv * slab_f4 (slab) and f - cc *
// slab_f4 < nv * wch_f4 (filters); with one channel per stage every stage is
// full.
__host__ __device__ inline bool mfma_slot_loads(const MfmaTile& T, const MfmaBlock& g, int f,
                                                int goff, int nv)
{
    if (T.CCT == 1) return f < g.total_f4;
    return goff >= 0 ? f < nv * g.slab_f4
                     : (f < g.total_f4 && f - g.cc * g.slab_f4 < nv * g.wch_f4);
}

// Float offsets from a.x / a.w of the block's slab and filter bases.
__host__ __device__ inline int64_t mfma_x_base(const MfmaTile& T, const MfmaArgs& a,
                                               const MfmaBlock& g)
{
    return ((int64_t)g.b0 * a.C_in * (T.KD == 3 ? g.D : 1) + g.z0) * g.plane_floats;
}
__host__ __device__ inline int64_t mfma_w_base(const MfmaTile& T, const MfmaBlock& g)
{
    return (int64_t)g.co0 * g.taps_full * T.NB;
}

// Channels of stage s: [ci0, ci0 + n_valid) of filter plane qz (k = 3).
__host__ __device__ inline int mfma_stage_channels(const MfmaTile& T, const MfmaArgs& a,
                                                   const MfmaBlock& g, int s, int& ci0, int& qz)
{
    int cg = s;
    qz = 0;
    if (T.KD == 3) {
        cg = udiv(s, g.df);
        qz = s - cg * g.df;
    }
    ci0 = cg * g.cc;
    return g.cc < a.C_in - ci0 ? g.cc : a.C_in - ci0;
}

// Offsets of stage (ci0, qz)'s slab and filter bases from the block's bases.
__host__ __device__ inline int64_t mfma_stage_x(const MfmaBlock& g, int ci0, int qz)
{
    return (int64_t)ci0 * g.x_cstride + (int64_t)qz * g.plane_floats;
}
__host__ __device__ inline int64_t mfma_stage_w(const MfmaTile& T, const MfmaBlock& g, int ci0,
                                                int qz)
{
    return (int64_t)ci0 * g.w_cstride + (int64_t)qz * g.taps2 * T.NB;
}

// LDS float offset where wave `wave` lands slot t of buffer buf: the wave's
// base in the buffer plus the slot's offset; a direct 16-byte global->LDS load
// puts lane i 4 i floats further.
__host__ __device__ inline int mfma_lds_wave(const MfmaArgs& a, int buf, int wave)
{
    return buf * a.stage_floats + wave * 256;
}
__host__ __device__ inline int mfma_lds_slot(const MfmaTile& T, int t) { return t * T.nt() * 4; }

// Per-lane fragment constants.  A (16 x 4): row mrow = (output channel co_a,
// output blade i_a), column kk = input blade j = 4 h + kk; the lane reads the
// raw filter blade src(i_a, j) and applies the table's sign.  B (4 x 16): row
// kk = input blade, column mrow = output position.
struct MfmaLane {
    int lane, wk, wrest, wco, wpos, mrow, kk;
};

__host__ __device__ inline MfmaLane mfma_lane(const MfmaTile& T, int tid)
{
    MfmaLane l;
    l.lane = tid & 63;
    const int wave = tid >> 6;
    l.wk = wave / (T.WCO * T.WPOS);  // K slice of this wave
    l.wrest = wave - l.wk * (T.WCO * T.WPOS);
    l.wco = l.wrest % T.WCO;
    l.wpos = l.wrest / T.WCO;
    l.mrow = l.lane & 15;
    l.kk = l.lane >> 4;
    return l;
}

// A fragment: buffer float offset of the lane's raw filter blade for blade
// group h (NEG: in the copy of the lane's sign), before the per-step part.
__host__ __device__ inline int mfma_a_ofs(const MfmaTile& T, const MfmaArgs& a,
                                          const MfmaBlock& g, const MfmaLane& l, int h)
{
    const int co_a = l.mrow / T.NB, i_a = l.mrow % T.NB;
    const bool neg = T.NEG && sign_of(a.sign, i_a * T.NB + 4 * h + l.kk) < 0.0f;
    return (neg ? g.w_neg : g.w_lds) + (l.wco * T.MW * T.cpt() + co_a) * g.taps2 * T.NB +
           src_blade(T.NB, i_a, 4 * h + l.kk);
}
__host__ __device__ inline float mfma_a_sign(const MfmaTile& T, const MfmaArgs& a,
                                             const MfmaLane& l, int h)
{
    const int i_a = l.mrow % T.NB;
    return sign_of(a.sign, i_a * T.NB + 4 * h + l.kk);
}
// per step: channel c of the stage (its filters start mfma_a_chan(wch_f4, c)
// floats into the buffer), then channel tile mw and filter tap (2D index) around the
// lane's offset (wtaps: taps per filter plane, d_filter^2)
__host__ __device__ inline int mfma_a_chan(int wch_f4, int c) { return c * wch_f4 * 4; }
__host__ __device__ inline int mfma_a_tap(const MfmaTile& T, int wtaps, int wofs, int mw, int tap)
{
    return wofs + mw * (T.cpt() * wtaps * T.NB) + tap * T.NB;
}

// B fragment: buffer float offset of the lane's input blade kk at output
// position column nw, before the per-step part (mfma_b_chan, mfma_b_tap).  Tail lanes
// read a valid position; their outputs are never stored.
__host__ __device__ inline int mfma_b_ofs(const MfmaTile& T, const MfmaBlock& g,
                                          const MfmaLane& l, int nw)
{
    const int Do = g.Do, D = g.D;
    int m = g.m0 + (l.wpos * T.NW + nw) * 16 + l.mrow;
    m = m < g.m_end - 1 ? m : g.m_end - 1;
    const int r = fdiv(m, g.fDo);
    const int xx = m - r * Do;
    const int pl = fdiv(r, g.fDo);
    const int yy = r - pl * Do;
    const int srow = pl == g.pl0 ? yy - g.ylo0 : g.len0 + (pl - g.pl0 - 1) * D + yy;
    return srow * g.lrow_floats + (xx - g.x0) * 4 + l.kk;
}
// per step: channel c (its slab starts mfma_b_chan(slab_f4, c) floats in),
// then filter row qy and column qx of the tap and blade group h around the
// lane's offset (lrow_floats, D: the block's LDS row stride and d_image)
__host__ __device__ inline int mfma_b_chan(int slab_f4, int c) { return c * slab_f4 * 4; }
__host__ __device__ inline int mfma_b_tap(int lrow_floats, int D, int xoff, int h, int qy, int qx)
{
    return xoff + qy * lrow_floats + h * D * 4 + qx * 4;
}

// K split: float4 index in LDS where K slice wk >= 1 leaves tile (mw, nw) of
// lane `lane` for slice 0.
__host__ __device__ inline int mfma_red_f4(const MfmaTile& T, int wk, int wrest, int mw, int nw,
                                           int lane)
{
    return ((wk - 1) * (T.WCO * T.WPOS * T.MW * T.NW) + (wrest * T.MW + mw) * T.NW + nw) * 64 +
           lane;
}

// Epilogue: a D fragment lane holds rows 4 kk + r of the tile, i.e. output
// channel co_o and blades i0 .. i0 + 3, for position column mrow.
__host__ __device__ inline int mfma_out_channel(const MfmaTile& T, const MfmaBlock& g,
                                                const MfmaLane& l, int mw)
{
    const int co_o = T.NB == 4 ? l.kk : (l.kk >> 1);
    return g.co0 + (l.wco * T.MW + mw) * T.cpt() + co_o;
}
__host__ __device__ inline int mfma_out_blade0(const MfmaTile& T, const MfmaLane& l)
{
    return T.NB == 4 ? 0 : 4 * (l.kk & 1);
}
__host__ __device__ inline int mfma_out_pos(const MfmaTile& T, const MfmaBlock& g,
                                            const MfmaLane& l, int nw)
{
    return g.m0 + (l.wpos * T.NW + nw) * 16 + l.mrow;
}
// float offset in the output of (position m, channel co, blade i0): stored
// when co < C_out and m < m_end
__host__ __device__ inline int64_t mfma_out_ofs(const MfmaTile& T, const MfmaArgs& a, int m,
                                                int co, int i0)
{
    const int b = udiv(m, a.npos);
    const int sp = m - b * a.npos;
    return (((int64_t)b * a.C_out + co) * a.npos + sp) * T.NB + i0;
}

}  // namespace cliff
