// Host-side walk of conv_mfma_kernel's address arithmetic (test
// infrastructure; see check_main.cpp).  Everything below calls the kernel's
// own functions from conv_mfma_geom.hpp.
//
// For a launch plan it checks:
//   * launch shape: workgroup size, grid = the number of blocks, LDS bytes
//     within the 160 KiB of a CU and holding two stage buffers (and the K
//     split's partial sums), every staged float4 inside its stage buffer;
//   * every workgroup: each lane's direct global->LDS loads (16 bytes) lie
//     inside the input or filter tensor, for the first stage, the last full
//     stage and the last stage (the offsets grow with the stage and the load
//     set depends only on the stage's channel count, so these bound every
//     stage); every output store (16 bytes, 16-byte aligned) lies inside the
//     output at the position and channel the lane holds, and every output
//     multivector is stored exactly once over the grid; bias reads in bounds;
//   * sampled workgroups (all of them on small grids): the LDS words written
//     by the stage are simulated, and every MFMA fragment read of every lane,
//     channel, tap and blade group must hit a word this stage wrote that
//     holds the input or filter element the product needs:
//       B: input[b, ci0 + c, p + q, 4 h + kk] for the lane's position p
//          (clamped to the block's last for tail lanes, never stored);
//       A: filters[ci0 + c, co, q, src(i, 4 h + kk)] for the lane's output
//          channel co and blade i (channels past C_out: the last channel).
#include <stdio.h>

#include <algorithm>
#include <vector>

#include "check.hpp"
#include "conv_mfma_geom.hpp"

namespace hostcheck {

using namespace cliff;

namespace {

struct Ctx {
    MfmaTile T;
    const MfmaArgs* a;
    int64_t lds_bytes;
    int64_t B, C_in, C_out, D, Do, df, npos, img;
    int64_t n_x, n_w, n_y, n_bias;
};

// spatial coordinates (k = 2: y, x; k = 3: z, y, x) of flat index sp over n^k
void unflat(int64_t sp, int k, int64_t n, int64_t* c)
{
    for (int t = k - 1; t >= 0; --t) {
        c[t] = sp % n;
        sp /= n;
    }
}

// Direct-load bounds and (optionally) the LDS image of one stage.
// lds_src[i]: -1 unwritten; else (kind << 60) | global float index, kind 1 =
// input, 2 = filters.
bool stage_loads(const Ctx& C, const MfmaBlock& g, int s, const std::vector<int>& goff,
                 std::vector<int64_t>* lds_src, int bid)
{
    const MfmaTile& T = C.T;
    const MfmaArgs& a = *C.a;
    const int NT = T.nt();
    int ci0, qz;
    const int nv = mfma_stage_channels(T, a, g, s, ci0, qz);
    if (nv < 1) {
        fail("block %d stage %d has %d channels", bid, s, nv);
        return false;
    }
    const int64_t xs = mfma_x_base(T, a, g) + mfma_stage_x(g, ci0, qz);
    const int64_t ws = mfma_w_base(T, g) + mfma_stage_w(T, g, ci0, qz);
    const int buf = s & 1;
    bool ok = true;
    for (int t = 0; t < T.SLOTS; ++t)
        for (int tid = 0; tid < NT; ++tid) {
            const int f = t * NT + tid;
            const int go = goff[(size_t)t * NT + tid];
            if (!mfma_slot_loads(T, g, f, go, nv)) continue;
            const bool is_x = go >= 0;
            const int64_t src = is_x ? xs + go : ws + (-1 - (int64_t)go);
            const int64_t n = is_x ? C.n_x : C.n_w;
            if (src < 0 || src + 4 > n || (src & 3)) {
                fail("block %d stage %d slot %d lane %d: %s load at float %lld of %lld",
                     bid, s, t, tid, is_x ? "input" : "filter", (long long)src, (long long)n);
                ok = false;
                continue;
            }
            const int64_t dst =
                mfma_lds_wave(a, buf, tid >> 6) + mfma_lds_slot(T, t) + 4 * (tid & 63);
            if (dst < (int64_t)buf * a.stage_floats || dst + 4 > (int64_t)(buf + 1) * a.stage_floats ||
                (dst + 4) * 4 > C.lds_bytes) {
                fail("block %d stage %d slot %d lane %d: LDS write at float %lld outside "
                     "stage buffer %d", bid, s, t, tid, (long long)dst, buf);
                ok = false;
                continue;
            }
            if (lds_src) {
                const int64_t base = dst - (int64_t)buf * a.stage_floats;
                for (int e = 0; e < 4; ++e) {
                    int64_t& slot = (*lds_src)[base + e];
                    if (slot != -1) {
                        fail("block %d stage %d: LDS float %lld written twice", bid, s,
                             (long long)(base + e));
                        ok = false;
                    }
                    slot = ((int64_t)(is_x ? 1 : 2) << 60) | (src + e);
                }
            }
        }
    // NEG: the filters again through registers, written negated
    for (int u = 0; u < T.fslots(); ++u)
        for (int tid = 0; tid < NT; ++tid) {
            const int e = u * NT + tid;
            if (e >= g.cc * g.wch_f4) continue;
            const int64_t src = ws + mfma_filter_src(T, a, g, e);
            if (src < 0 || src + 4 > C.n_w || (src & 3)) {
                fail("block %d stage %d filter register %d lane %d: load at float %lld of %lld",
                     bid, s, u, tid, (long long)src, (long long)C.n_w);
                ok = false;
                continue;
            }
            for (int neg = 1; neg < 2; ++neg) {  // the negated copy (the other: direct loads)
                const int64_t dst = mfma_wreg_lds(g, e, neg);
                if (dst < 0 || dst + 4 > a.stage_floats ||
                    ((int64_t)buf * a.stage_floats + dst + 4) * 4 > C.lds_bytes) {
                    fail("block %d stage %d filter register %d lane %d: LDS write at %lld",
                         bid, s, u, tid, (long long)dst);
                    ok = false;
                    continue;
                }
                if (!lds_src) continue;
                for (int q = 0; q < 4; ++q) {
                    int64_t& slot = (*lds_src)[dst + q];
                    if (slot != -1) {
                        fail("block %d stage %d: LDS float %lld written twice", bid, s,
                             (long long)(dst + q));
                        ok = false;
                    }
                    slot = ((int64_t)(neg ? 3 : 2) << 60) | (src + q);
                }
            }
        }
    return ok;
}

int64_t x_index(const Ctx& C, int64_t b, int64_t ci, const int64_t* sp, int j)
{
    int64_t f = 0;
    for (int t = 0; t < C.T.KD; ++t) f = f * C.D + sp[t];
    return ((b * C.C_in + ci) * C.img + f) * C.T.NB + j;
}

int64_t w_index(const Ctx& C, int64_t ci, int64_t co, const int* q, int blade)
{
    int64_t f = 0;
    for (int t = 0; t < C.T.KD; ++t) f = f * C.df + q[t];
    int64_t taps = 1;
    for (int t = 0; t < C.T.KD; ++t) taps *= C.df;
    return ((ci * C.C_out + co) * taps + f) * C.T.NB + blade;
}

// Every fragment read of every lane for stage s against the simulated LDS.
void stage_fragments(const Ctx& C, const MfmaBlock& g, int s, const std::vector<int64_t>& lds_src,
                     int bid)
{
    const MfmaTile& T = C.T;
    const MfmaArgs& a = *C.a;
    const int NT = T.nt(), NB = T.NB;
    int ci0, qz;
    const int nv = mfma_stage_channels(T, a, g, s, ci0, qz);
    const int df = g.df;
    int reported = 0;
    auto bad = [&](const char* what, int tid, int c, int tap, int h, int idx, int64_t ofs,
                   int64_t got, int64_t want) {
        if (reported++ < 2)
            fail("block %d stage %d lane %d channel %d tap %d group %d %s %d: LDS float %lld "
                 "holds %llx, needs %llx", bid, s, tid, c, tap, h, what, idx, (long long)ofs,
                 (unsigned long long)got, (unsigned long long)want);
    };
    for (int tid = 0; tid < NT; ++tid) {
        const MfmaLane L = mfma_lane(T, tid);
        const int co_a = L.mrow / NB, i_a = L.mrow % NB;
        for (int c = 0; c < nv; ++c)
            for (int tap = 0; tap < df * df; ++tap) {
                const int qy = tap / df, qx = tap % df;
                for (int h = 0; h < T.nh(); ++h) {
                    const int j = 4 * h + L.kk;
                    // A fragments
                    for (int mw = 0; mw < T.MW; ++mw) {
                        const int64_t ofs =
                            mfma_a_chan(g.wch_f4, c) +
                            mfma_a_tap(T, g.taps2, mfma_a_ofs(T, a, g, L, h), mw, tap);
                        int co = g.co0 + (L.wco * T.MW + mw) * T.cpt() + co_a;
                        if (co >= C.C_out) co = (int)C.C_out - 1;
                        int q[3];
                        if (T.KD == 2) {
                            q[0] = qy;
                            q[1] = qx;
                        } else {
                            q[0] = qz;
                            q[1] = qy;
                            q[2] = qx;
                        }
                        // kind 3: the negated copy, read by lanes of sign -1 (NEG)
                        const int64_t kind = T.NEG && mfma_a_sign(T, a, L, h) < 0.f ? 3 : 2;
                        const int64_t want =
                            (kind << 60) | w_index(C, ci0 + c, co, q, src_blade(NB, i_a, j));
                        const int64_t got =
                            ofs >= 0 && ofs < (int64_t)lds_src.size() ? lds_src[ofs] : -2;
                        if (got != want) bad("A tile", tid, c, tap, h, mw, ofs, got, want);
                    }
                    // B fragments
                    for (int nw = 0; nw < T.NW; ++nw) {
                        const int64_t ofs =
                            mfma_b_chan(g.slab_f4, c) +
                            mfma_b_tap(g.lrow_floats, g.D, mfma_b_ofs(T, g, L, nw), h, qy, qx);
                        int64_t m = g.m0 + (L.wpos * T.NW + nw) * 16 + L.mrow;
                        m = std::min<int64_t>(m, g.m_end - 1);
                        const int64_t b = m / C.npos;
                        int64_t sp[3];
                        unflat(m - b * C.npos, T.KD, C.Do, sp);
                        if (T.KD == 2) {
                            sp[0] += qy;
                            sp[1] += qx;
                        } else {
                            sp[0] += qz;
                            sp[1] += qy;
                            sp[2] += qx;
                        }
                        const int64_t want = ((int64_t)1 << 60) | x_index(C, b, ci0 + c, sp, j);
                        const int64_t got =
                            ofs >= 0 && ofs < (int64_t)lds_src.size() ? lds_src[ofs] : -2;
                        if (got != want) bad("B tile", tid, c, tap, h, nw, ofs, got, want);
                    }
                }
            }
    }
}

}  // namespace

void check_conv_mfma(const LaunchPlan& p)
{
    Ctx C;
    C.T = MfmaTile{p.tpl[0], p.tpl[1], p.tpl[2], p.tpl[3], p.tpl[4], p.tpl[5],
                   p.tpl[6], p.tpl[7], p.tpl[8], p.tpl[10], p.tpl[11]};
    const MfmaTile& T = C.T;
    const MfmaArgs& a = *static_cast<const MfmaArgs*>(p.args);
    C.a = &a;
    C.lds_bytes = p.lds_bytes;
    const Buffer* bx = find_buffer(a.x);
    const Buffer* bw = find_buffer(a.w);
    const Buffer* by = find_buffer(a.y);
    const Buffer* bb = a.bias ? find_buffer(a.bias) : nullptr;
    if (!bx || !bw || !by || (a.bias && !bb)) {
        fail("conv_mfma launch with a pointer that is no buffer of the call");
        return;
    }
    C.n_x = bx->n;
    C.n_w = bw->n;
    C.n_y = by->n;
    C.n_bias = bb ? bb->n : 0;
    C.C_in = a.C_in;
    C.C_out = a.C_out;
    C.D = a.D;
    C.Do = a.Do;
    C.df = a.df;
    C.npos = a.npos;
    C.img = 1;
    int64_t npos = 1;
    for (int t = 0; t < T.KD; ++t) {
        C.img *= C.D;
        npos *= C.Do;
    }
    C.B = a.M / std::max<int64_t>(1, a.npos);
    const int NT = T.nt(), NB = T.NB;

    // launch shape
    if (p.block != NT) fail("workgroup of %lld threads, the tile needs %d", (long long)p.block, NT);
    if (p.grid != a.n_blk || p.grid < 1) fail("grid %lld, %d blocks", (long long)p.grid, a.n_blk);
    if (npos != a.npos || (int64_t)a.M != C.B * npos) fail("position count mismatch");
    if (C.n_x != C.B * C.C_in * C.img * NB || C.n_y != C.B * C.C_out * npos * NB)
        fail("tensor sizes do not match the arguments");
    if (p.lds_bytes > 160 * 1024) fail("%lld LDS bytes exceed a CU's 160 KiB", (long long)p.lds_bytes);
    if (2 * (int64_t)a.stage_floats * 4 > p.lds_bytes)
        fail("two stage buffers (%d floats) exceed the %lld LDS bytes", a.stage_floats,
             (long long)p.lds_bytes);
    const int64_t red_bytes = (int64_t)(T.WK - 1) * T.WCO * T.WPOS * T.MW * T.NW * 64 * 16;
    if (red_bytes > p.lds_bytes) fail("K-split partial sums exceed the LDS");
    if (a.n_stage < 1) fail("no stage");
    if (p.grid < 1 || current->errors >= 8) return;

    // sampled workgroups for the LDS simulation: all on small grids
    const int64_t per_block = (int64_t)NT * a.cc * a.df * a.df * (T.MW + T.NW) * T.nh();
    const int64_t budget = 6000000;  // fragment reads simulated per launch (besides 16 blocks)
    const int64_t stride = std::max<int64_t>(1, (p.grid * per_block * 2) / budget);

    std::vector<uint8_t> written((size_t)(C.n_y / 4), 0);
    current->grid_sampled |= (p.grid >> 15) > 1;
    std::vector<int> goff((size_t)T.SLOTS * NT);
    std::vector<int64_t> lds_src;
    // grids of more than 2^15 workgroups: every (grid / 2^15)-th one, the
    // first and the last 64 (and no output coverage count)
    const int64_t wstride = std::max<int64_t>(1, p.grid >> 15);
    for (int bid = 0; bid < p.grid; ++bid) {
        if (wstride > 1 && bid % wstride && bid >= 64 && bid < p.grid - 64) continue;
        const MfmaBlock g = mfma_block(T, a, bid);
        if (g.m0 < 0 || g.m_end > a.M || g.m0 >= g.m_end || g.co0 < 0 || g.co0 >= a.C_out) {
            fail("block %d covers positions [%d, %d) of %d, channels from %d", bid, g.m0, g.m_end,
                 a.M, g.co0);
            continue;
        }
        if ((int64_t)g.total_f4 * 4 > a.stage_floats || (int64_t)T.SLOTS * NT < g.total_f4 ||
            (T.NEG && (g.cc != 1 || (int64_t)T.fslots() * NT < g.wch_f4 ||
                       g.w_neg + g.cc * g.wch_f4 * 4 > a.stage_floats)))
            fail("block %d stages %d float4 in %d slots of a %d-float buffer", bid, g.total_f4,
                 T.SLOTS * NT, a.stage_floats);
        for (int t = 0; t < T.SLOTS; ++t)
            for (int tid = 0; tid < NT; ++tid)
                goff[(size_t)t * NT + tid] = mfma_slot_goff(T, a, g, t * NT + tid);
        // stages that bound all: first, last full, last (3D: also the first
        // channel group's last plane)
        std::vector<int> stages = {0, a.n_stage - 1};
        for (int s = a.n_stage - 1; s >= 0; --s) {
            int ci0, qz;
            if (mfma_stage_channels(T, a, g, s, ci0, qz) == g.cc) {
                stages.push_back(s);
                break;
            }
        }
        if (T.KD == 3 && g.df - 1 < a.n_stage) stages.push_back(g.df - 1);
        std::sort(stages.begin(), stages.end());
        stages.erase(std::unique(stages.begin(), stages.end()), stages.end());
        const bool sim = bid % stride == 0 || bid < 8 || bid >= p.grid - 8;
        for (int s : stages) {
            // the LDS image of the first and the last stage
            const bool sim_s = sim && (s == 0 || s == a.n_stage - 1);
            if (sim_s) lds_src.assign((size_t)a.stage_floats, -1);
            if (stage_loads(C, g, s, goff, sim_s ? &lds_src : nullptr, bid) && sim_s)
                stage_fragments(C, g, s, lds_src, bid);
        }
        if (sim) current->workgroups++;

        // outputs and bias
        for (int tid = 0; tid < NT; ++tid) {
            const MfmaLane L = mfma_lane(T, tid);
            if (L.wk > 0) {
                for (int mw = 0; mw < T.MW; ++mw)
                    for (int nw = 0; nw < T.NW; ++nw) {
                        const int64_t r = mfma_red_f4(T, L.wk, L.wrest, mw, nw, L.lane);
                        if (r < 0 || (r + 1) * 16 > p.lds_bytes)
                            fail("block %d lane %d: partial sum at LDS float4 %lld", bid, tid,
                                 (long long)r);
                    }
                continue;  // K slices > 0 store nothing
            }
            const int i0 = mfma_out_blade0(T, L);
            for (int mw = 0; mw < T.MW; ++mw) {
                const int co = mfma_out_channel(T, g, L, mw);
                if (co >= a.C_out) continue;
                if (a.bias && ((int64_t)co * NB + i0 + 4 > C.n_bias))
                    fail("block %d lane %d: bias read past the bias", bid, tid);
                for (int nw = 0; nw < T.NW; ++nw) {
                    const int m = mfma_out_pos(T, g, L, nw);
                    if (m >= g.m_end) continue;
                    const int64_t ofs = mfma_out_ofs(T, a, m, co, i0);
                    const int64_t b = m / npos, sp = m - (m / npos) * npos;
                    const int64_t want = ((b * C.C_out + co) * npos + sp) * NB + i0;
                    if (ofs != want || ofs < 0 || ofs + 4 > C.n_y || (ofs & 3)) {
                        fail("block %d lane %d tile (%d, %d): store at float %lld, position %d "
                             "channel %d needs %lld", bid, tid, mw, nw, (long long)ofs, m, co,
                             (long long)want);
                        continue;
                    }
                    uint8_t& w = written[(size_t)(ofs / 4)];
                    if (w) fail("block %d lane %d: output float %lld stored twice", bid, tid,
                                (long long)ofs);
                    w = 1;
                }
            }
        }
        if (current->errors >= 8) return;
    }
    for (size_t i = 0; wstride == 1 && i < written.size(); ++i)
        if (!written[i]) {
            fail("output float %lld never stored", (long long)(i * 4));
            break;
        }
}

}  // namespace hostcheck
