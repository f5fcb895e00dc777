// Host-side walk of conv1d_mfma_kernel's address arithmetic (test
// infrastructure; see check_main.cpp), calling the kernel's own functions
// from conv1d_geom.hpp.
//
// For a launch plan it checks the launch shape (workgroup size, grid, LDS
// within a CU and holding two stage buffers and the K split's partial sums)
// and, per workgroup:
//   * every direct global->LDS load of every lane (FX / FW floats) inside the
//     input or filter tensor, aligned to its size, for the first, the last
//     full and the last stage (offsets grow with the stage, the load set
//     depends only on its channel count), landing inside its stage buffer's
//     window or filter section;
//   * sampled workgroups (all on small grids): the stage's LDS image, and
//     every fragment read of every lane, channel pair and tap hitting a word
//     the stage wrote with the element the product needs,
//       B: input[b, ci0 + c_l + c_sub, x + tap, j] for the lane's position,
//       A: filters[ci0 + c_l + c_sub, co, tap, src(i, j)] (channels past
//          C_out: any word of the buffer, their rows are never stored),
//     except the second channel of a masked pair (an odd channel count),
//     whose reads must only stay inside the buffer;
//   * every output store (8 bytes) inside the output at the lane's position
//     and channel, every output multivector stored once over the grid.
#include <stdio.h>

#include <algorithm>
#include <vector>

#include "check.hpp"
#include "conv1d_geom.hpp"

namespace hostcheck {

using namespace cliff;

namespace {

struct Ctx1 {
    C1Tile T;
    const C1Args* a;
    int64_t lds_bytes, n_x, n_w, n_y, n_bias, B;
};

bool stage1(const Ctx1& C, const C1Block& g, int s, const std::vector<uint32_t>& xoffb,
            const std::vector<uint32_t>& woffb, std::vector<int64_t>* lds, int bid)
{
    const C1Tile& T = C.T;
    const C1Args& a = *C.a;
    const int NT = T.nt();
    const int nv = c1_stage_channels(a, s);
    if (nv < 1) {
        fail("conv1d block %d stage %d has %d channels", bid, s, nv);
        return false;
    }
    const int64_t xs = c1_x_base(a, g) + c1_stage_x(a, s);
    const int64_t ws = c1_w_base(g) + c1_stage_w(a, g, s);
    const int buf = s & 1;
    const int64_t b0 = (int64_t)buf * a.stage_floats, b1 = b0 + a.stage_floats;
    bool ok = true;
    auto put = [&](int64_t dst, int n, int kind, int64_t src) {
        if (!lds) return;
        for (int e = 0; e < n; ++e) {
            int64_t& slot = (*lds)[dst - b0 + e];
            if (slot != -1) {
                fail("conv1d block %d stage %d: LDS float %lld written twice", bid, s,
                     (long long)(dst - b0 + e));
                ok = false;
            }
            slot = ((int64_t)kind << 60) | (src + e);
        }
    };
    for (int t = 0; t < T.SIN; ++t)
        for (int tid = 0; tid < NT; ++tid) {
            const int f = (t * NT + tid) * T.FX;
            if (!c1_x_loads(a, f, nv)) continue;
            const int64_t src = xs + xoffb[(size_t)t * NT + tid] / 4;
            const int64_t dst = c1_lds_x(T, a, buf, t, tid >> 6) + (int64_t)T.FX * (tid & 63);
            if (src < 0 || src + T.FX > C.n_x || src % T.FX) {
                fail("conv1d block %d stage %d input slot %d lane %d: load at float %lld of %lld",
                     bid, s, t, tid, (long long)src, (long long)C.n_x);
                ok = false;
                continue;
            }
            if (dst < b0 || dst + T.FX > b0 + (int64_t)a.ccp * a.span2) {
                fail("conv1d block %d stage %d input slot %d lane %d: LDS write at %lld outside "
                     "the windows", bid, s, t, tid, (long long)dst);
                ok = false;
                continue;
            }
            put(dst, T.FX, 1, src);
        }
    for (int t = 0; t < T.SW; ++t)
        for (int tid = 0; tid < NT; ++tid) {
            const int e = (t * NT + tid) * T.FW;
            const uint32_t wo = woffb[(size_t)t * NT + tid];
            if (!c1_w_loads(T, g, e, wo, nv)) continue;
            const int64_t src = ws + wo / 4;
            const int64_t dst = c1_lds_w(T, a, g, buf, t, tid >> 6) + (int64_t)T.FW * (tid & 63);
            if (src < 0 || src + T.FW > C.n_w || src % T.FW) {
                fail("conv1d block %d stage %d filter slot %d lane %d: load at float %lld of %lld",
                     bid, s, t, tid, (long long)src, (long long)C.n_w);
                ok = false;
                continue;
            }
            if (dst < b0 + g.w_lds || dst + T.FW > b1 || (dst + T.FW) * 4 > C.lds_bytes) {
                fail("conv1d block %d stage %d filter slot %d lane %d: LDS write at %lld outside "
                     "the filters", bid, s, t, tid, (long long)dst);
                ok = false;
                continue;
            }
            put(dst, T.FW, 2, src);
        }
    return ok;
}

void fragments1(const Ctx1& C, const C1Block& g, int s, const std::vector<int64_t>& lds, int bid)
{
    const C1Tile& T = C.T;
    const C1Args& a = *C.a;
    const int NT = T.nt(), df = g.df;
    const int nv = c1_stage_channels(a, s), ci0 = s * a.cc;
    int reported = 0;
    for (int tid = 0; tid < NT; ++tid) {
        const C1Lane L = c1_lane(T, tid);
        const int co_a = L.mrow >> 1, i_a = L.mrow & 1;
        const int wofs = c1_a_ofs(T, g, L);
        for (int c_l = 0; c_l < nv; c_l += 2) {
            const bool masked = c_l + 1 >= nv && L.c_sub == 1;  // the missing channel
            const int ci = ci0 + c_l + L.c_sub;
            for (int tap = 0; tap < df; ++tap) {
                for (int mw = 0; mw < T.MW; ++mw) {
                    const int64_t ofs = c1_a_pair(g, c_l) + c1_a_step(g, wofs, mw, tap);
                    const int co = g.co0 + (L.wco * T.MW + mw) * 8 + co_a;
                    if (ofs < 0 || ofs >= a.stage_floats) {
                        if (reported++ < 2)
                            fail("conv1d block %d lane %d: A read at %lld outside the buffer",
                                 bid, tid, (long long)ofs);
                        continue;
                    }
                    if (masked || co >= a.C_out) continue;
                    const int64_t want =
                        ((int64_t)2 << 60) |
                        ((((int64_t)ci * a.C_out + co) * df + tap) * 2 + src_blade(2, i_a, L.j));
                    if (lds[ofs] != want && reported++ < 2)
                        fail("conv1d block %d stage %d lane %d pair %d tap %d A %d: LDS %lld holds "
                             "%llx, needs %llx", bid, s, tid, c_l, tap, mw, (long long)ofs,
                             (unsigned long long)lds[ofs], (unsigned long long)want);
                }
                for (int nw = 0; nw < T.NW; ++nw) {
                    const int64_t ofs = c1_b_pair(a, c_l) + c1_b_ofs(T, a, g, L, nw) + 2 * tap;
                    if (ofs < 0 || ofs >= a.stage_floats) {
                        if (reported++ < 2)
                            fail("conv1d block %d lane %d: B read at %lld outside the buffer",
                                 bid, tid, (long long)ofs);
                        continue;
                    }
                    if (masked) continue;
                    int m = g.m0 + (L.wpos * T.NW + nw) * 16 + L.mrow;
                    m = std::min(m, g.m_end - 1);
                    const int64_t b = m / a.Do, x = m - b * a.Do + tap;
                    const int64_t want = ((int64_t)1 << 60) |
                                         (((b * a.C_in + ci) * a.D + x) * 2 + L.j);
                    if (lds[ofs] != want && reported++ < 2)
                        fail("conv1d block %d stage %d lane %d pair %d tap %d B %d: LDS %lld holds "
                             "%llx, needs %llx", bid, s, tid, c_l, tap, nw, (long long)ofs,
                             (unsigned long long)lds[ofs], (unsigned long long)want);
                }
            }
        }
    }
}

}  // namespace

void check_conv1d(const LaunchPlan& p)
{
    Ctx1 C;
    // <DF, WCO, WPOS, MW, NW, SIN, SW, WAVES, FW, FX, WK>
    C.T = C1Tile{p.tpl[0], p.tpl[1], p.tpl[2], p.tpl[3], p.tpl[4],
                 p.tpl[5], p.tpl[6], p.tpl[8], p.tpl[9], p.tpl[10]};
    const C1Tile& T = C.T;
    const C1Args& a = *static_cast<const C1Args*>(p.args);
    C.a = &a;
    C.lds_bytes = p.lds_bytes;
    const Buffer* bx = find_buffer(a.x);
    const Buffer* bw = find_buffer(a.w);
    const Buffer* by = find_buffer(a.y);
    const Buffer* bb = a.bias ? find_buffer(a.bias) : nullptr;
    if (!bx || !bw || !by || (a.bias && !bb)) {
        fail("conv1d launch with a pointer that is no buffer of the call");
        return;
    }
    C.n_x = bx->n;
    C.n_w = bw->n;
    C.n_y = by->n;
    C.n_bias = bb ? bb->n : 0;
    C.B = a.M / a.Do;
    const int NT = T.nt();
    if (p.block != NT) fail("conv1d: workgroup of %lld threads, the tile needs %d",
                            (long long)p.block, NT);
    if (p.grid != a.n_blk || p.grid < 1) fail("conv1d: grid %lld, %d blocks", (long long)p.grid,
                                              a.n_blk);
    if (C.n_x != C.B * a.C_in * a.D * 2 || C.n_y != C.B * a.C_out * a.Do * 2)
        fail("conv1d: tensor sizes do not match the arguments");
    if (p.lds_bytes > 160 * 1024 || 2 * (int64_t)a.stage_floats * 4 > p.lds_bytes)
        fail("conv1d: LDS %lld bytes for two %d-float buffers", (long long)p.lds_bytes,
             a.stage_floats);
    if ((int64_t)a.ccp * a.span2 + (int64_t)a.ccp * T.co_wg() * a.df * 2 > a.stage_floats)
        fail("conv1d: stage sections exceed the stage buffer");
    if ((int64_t)(T.WK - 1) * T.WCO * T.WPOS * T.MW * T.NW * 64 * 16 > p.lds_bytes)
        fail("conv1d: K-split partial sums exceed the LDS");
    if (current->errors >= 8 || p.grid < 1) return;

    const int64_t per_block = (int64_t)NT * a.cc / 2 * a.df * (T.MW + T.NW);
    const int64_t stride = std::max<int64_t>(1, (p.grid * per_block * 2) / 6000000);
    const int64_t wstride = std::max<int64_t>(1, p.grid >> 15);
    current->grid_sampled |= wstride > 1;
    std::vector<uint8_t> written((size_t)(C.n_y / 2), 0);
    std::vector<uint32_t> xoffb((size_t)T.SIN * NT), woffb((size_t)T.SW * NT);
    std::vector<int64_t> lds;
    for (int bid = 0; bid < p.grid; ++bid) {
        if (wstride > 1 && bid % wstride && bid >= 64 && bid < p.grid - 64) continue;
        const C1Block g = c1_block(T, a, bid);
        if (g.m0 < 0 || g.m_end > a.M || g.m0 >= g.m_end || g.co0 >= a.C_out ||
            g.span * 2 > a.span2) {
            fail("conv1d block %d: positions [%d, %d) of %d, window %d positions in %d floats",
                 bid, g.m0, g.m_end, a.M, g.span, a.span2);
            continue;
        }
        for (int t = 0; t < T.SIN; ++t)
            for (int tid = 0; tid < NT; ++tid)
                xoffb[(size_t)t * NT + tid] = c1_xoffb(T, a, g, (t * NT + tid) * T.FX);
        for (int t = 0; t < T.SW; ++t)
            for (int tid = 0; tid < NT; ++tid)
                woffb[(size_t)t * NT + tid] = c1_woffb(T, a, g, (t * NT + tid) * T.FW);
        std::vector<int> stages = {0, a.n_stage - 1};
        for (int s = a.n_stage - 1; s >= 0; --s)
            if (c1_stage_channels(a, s) == a.cc) {
                stages.push_back(s);
                break;
            }
        std::sort(stages.begin(), stages.end());
        stages.erase(std::unique(stages.begin(), stages.end()), stages.end());
        const bool sim = bid % stride == 0 || bid < 8 || bid >= p.grid - 8;
        for (int s : stages) {
            const bool sim_s = sim && (s == 0 || s == a.n_stage - 1);
            if (sim_s) lds.assign((size_t)a.stage_floats, -1);
            if (stage1(C, g, s, xoffb, woffb, sim_s ? &lds : nullptr, bid) && sim_s)
                fragments1(C, g, s, lds, bid);
        }
        if (sim) current->workgroups++;
        for (int tid = 0; tid < NT; ++tid) {
            const C1Lane L = c1_lane(T, tid);
            if (L.wk > 0) {
                for (int mw = 0; mw < T.MW; ++mw)
                    for (int nw = 0; nw < T.NW; ++nw) {
                        const int64_t r = c1_red_f4(T, L.wk, L.wrest, mw, nw, L.lane);
                        if (r < 0 || (r + 1) * 16 > p.lds_bytes)
                            fail("conv1d block %d lane %d: partial sum at LDS float4 %lld", bid,
                                 tid, (long long)r);
                    }
                continue;
            }
            for (int mw = 0; mw < T.MW; ++mw)
                for (int half = 0; half < 2; ++half) {
                    const int co = c1_out_channel(T, g, L, mw, half);
                    if (co >= a.C_out) continue;
                    if (a.bias && (int64_t)co * 2 + 2 > C.n_bias)
                        fail("conv1d block %d lane %d: bias read past the bias", bid, tid);
                    for (int nw = 0; nw < T.NW; ++nw) {
                        const int m = c1_out_pos(T, g, L, nw);
                        if (m >= g.m_end) continue;
                        const int64_t ofs = c1_out_base(a, m) + c1_out_chan(a, co);
                        const int64_t b = m / a.Do, x = m - b * a.Do;
                        const int64_t want = ((b * a.C_out + co) * a.Do + x) * 2;
                        if (ofs != want || ofs + 2 > C.n_y || (ofs & 1)) {
                            fail("conv1d block %d lane %d: store at %lld, needs %lld", bid, tid,
                                 (long long)ofs, (long long)want);
                            continue;
                        }
                        uint8_t& w = written[(size_t)(ofs / 2)];
                        if (w) fail("conv1d block %d lane %d: output float %lld stored twice",
                                    bid, tid, (long long)ofs);
                        w = 1;
                    }
                }
        }
        if (current->errors >= 8) return;
    }
    for (size_t i = 0; wstride == 1 && i < written.size(); ++i)
        if (!written[i]) {
            fail("conv1d: output float %lld never stored", (long long)(i * 2));
            break;
        }
}

}  // namespace hostcheck
