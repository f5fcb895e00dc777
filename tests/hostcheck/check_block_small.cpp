// Host-side walk of block_small_kernel's address arithmetic (test
// infrastructure; see check_main.cpp), calling the kernel's own functions
// from block_small_geom.hpp.
//
// For a launch plan it checks the launch shape and the LDS layout (input
// band, intermediate band and both filter areas disjoint and inside the
// launch's LDS) and, per workgroup (every one on grids of at most 2^15,
// else a sample):
//   * every direct global->LDS load of the input band and both filter
//     tensors inside its tensor, 16-byte aligned, landing inside its area;
//   * every fragment read of every lane, tile, input channel, tap and blade
//     group hitting the LDS word that holds the element the product needs:
//       layer 1 B: input[b, ci, s0 + so + qs, (yy + qy,) xx + qx, j],
//       layer 2 B: the intermediate word layer 1 stored for (ci, so + qs,
//                  (yy + qy,) xx + qx, j), which must have been stored,
//       A: filters[ci, co, tap, src(i, j)] of the layer;
//   * the epilogue's parameter loads (bias, Linear gate weight and bias, or
//     the input's first floats where a parameter is absent) in bounds;
//   * every intermediate store inside its area and made once per band, every
//     output store inside the output at its position, every output
//     multivector stored once over the grid.
#include <stdio.h>

#include <vector>

#include "block_small_geom.hpp"
#include "check.hpp"

namespace hostcheck {

using namespace cliff;

namespace {

int64_t buf_n(const void* p)
{
    const Buffer* b = find_buffer(p);
    return b ? b->n : -1;
}

}  // namespace

void check_block_small(const LaunchPlan& p)
{
    const BlockArgs& a = *static_cast<const BlockArgs*>(p.args);
    const int KD = p.tpl[0], NB = p.tpl[1], DFT = p.tpl[2];
    const int df = DFT > 0 ? DFT : a.df;
    const int NH = NB / 4;
    if (p.block != 256) fail("block_small: workgroup of %lld threads", (long long)p.block);
    if (p.lds_bytes > 160 * 1024) fail("block_small: %lld LDS bytes", (long long)p.lds_bytes);
    if (KD < 2 || KD > 3 || NB != (1 << KD) || df < 1 || a.taps != bs_ipow(df, KD))
        fail("block_small: k %d, N_B %d, d_filter %d, taps %d", KD, NB, df, a.taps);
    const int64_t n_x = buf_n(a.x), n_w1 = buf_n(a.w1), n_w2 = buf_n(a.w2), n_y = buf_n(a.y);
    if (n_x < 0 || n_w1 < 0 || n_w2 < 0 || n_y < 0) {
        fail("block_small: a tensor pointer is not a case buffer");
        return;
    }
    if (a.D1 != a.D0 - df + 1 || a.D2 != a.D1 - df + 1 || a.D2 < 1)
        fail("block_small: sizes %d -> %d -> %d with d_filter %d", a.D0, a.D1, a.D2, df);
    if (n_x != (int64_t)(p.grid / a.n_band) * a.C0 * bs_ipow(a.D0, KD) * NB ||
        n_y != (int64_t)(p.grid / a.n_band) * a.C2 * bs_ipow(a.D2, KD) * NB ||
        (int64_t)a.n_band * a.R < a.D2 || (int64_t)(a.n_band - 1) * a.R >= a.D2 ||
        p.grid % a.n_band)
        fail("block_small: grid %lld of %d bands x %d slices against the tensors",
             (long long)p.grid, a.n_band, a.R);
    if (current->errors) return;

    const int taps = a.taps;
    const int64_t lds_floats = p.lds_bytes / 4;
    const int n1 = a.C0 * a.C1 * taps * NB, n2 = a.C1 * a.C2 * taps * NB;
    if (n1 != n_w1 || n2 != n_w2) fail("block_small: filter sizes");
    // the largest band fixes the areas' extents
    const BsBand g0 = bs_band(a, KD, df, 0);
    const int64_t band_f = (int64_t)a.C0 * bs_band_f4(g0, NB) * 4;
    const int64_t y1_f = (int64_t)a.C1 * g0.R1 * g0.S1 * NB;
    if (!(band_f <= a.lds_y1 && a.lds_y1 + y1_f <= a.lds_w1 && a.lds_w1 + n1 <= a.lds_w2 &&
          a.lds_w2 + n2 <= lds_floats && a.lds_w1 % 4 == 0 && a.lds_w2 % 4 == 0 &&
          a.lds_y1 % 4 == 0))
        fail("block_small: LDS areas band %lld, y1 %d+%lld, w1 %d+%d, w2 %d+%d in %lld floats",
             (long long)band_f, a.lds_y1, (long long)y1_f, a.lds_w1, n1, a.lds_w2, n2,
             (long long)lds_floats);
    if (current->errors) return;

    const int64_t n_b1 = a.b1 ? buf_n(a.b1) : 0, n_b2 = a.b2 ? buf_n(a.b2) : 0;
    std::vector<uint8_t> written((size_t)(n_y / 4), 0);
    const int64_t wstride = std::max<int64_t>(1, p.grid >> 15);
    current->grid_sampled |= wstride > 1;
    std::vector<int64_t> band_src;  // input float held by each band LDS float
    std::vector<uint8_t> y1_set;
    for (int64_t bid = 0; bid < p.grid; ++bid) {
        if (wstride > 1 && bid % wstride && bid >= 64 && bid < p.grid - 64) continue;
        const BsBand g = bs_band(a, KD, df, (int)bid);
        if (g.R2 < 1 || g.s0 + g.R2 > a.D2 || g.b * a.n_band + g.s0 / a.R != bid) {
            fail("block_small block %lld: band b %d slices %d+%d", (long long)bid, g.b, g.s0,
                 g.R2);
            continue;
        }
        // 1. staging
        const int nx4 = a.C0 * bs_band_f4(g, NB);
        band_src.assign((size_t)nx4 * 4, -1);
        for (int e = 0; e < nx4; ++e) {
            const int64_t src = bs_band_src(a, g, NB, e);
            if (src < 0 || src + 4 > n_x || (src & 3)) {
                fail("block_small block %lld: band float4 %d from input float %lld of %lld",
                     (long long)bid, e, (long long)src, (long long)n_x);
                break;
            }
            for (int q = 0; q < 4; ++q) band_src[(size_t)4 * e + q] = src + q;
        }
        if (current->errors >= 8) return;

        // 2. both layers
        y1_set.assign((size_t)y1_f, 0);
        for (int li = 0; li < 2; ++li) {
            const BsLayer L = li == 0 ? bs_layer1(a, g) : bs_layer2(a, g);
            const int in_area = li == 0 ? nx4 * 4 : a.C1 * g.R1 * g.S1 * NB;
            const int w_area = li == 0 ? n1 : n2;
            const float* bias = li == 0 ? a.b1 : a.b2;
            const int64_t n_bias = li == 0 ? n_b1 : n_b2;
            const ActParams& act = li == 0 ? a.act1 : a.act2;
            const int npos = L.Rout * L.Sout;
            const int T = bs_tiles(L, NB);
            const int nrt = KD == 3 ? df * df : df;
            for (int t = 0; t < T; ++t) {
                for (int lane = 0; lane < 64; ++lane) {
                    const BsLane ln = bs_lane(NB, lane);
                    const BsTile tl = bs_tile(L, KD, NB, taps, ln, t);
                    if (tl.co_r < 0 || tl.co_r >= L.Cout || tl.m_r < 0 || tl.m_r >= npos) {
                        fail("block_small block %lld layer %d tile %d lane %d: row %d column %d",
                             (long long)bid, li + 1, t, lane, tl.co_r, tl.m_r);
                        continue;
                    }
                    for (int ci = 0; ci < L.Cin; ++ci)
                        for (int qs = 0; qs < df; ++qs)
                            for (int u = 0; u < nrt; ++u) {
                                const int qy = KD == 3 ? u / df : 0;
                                const int qx = KD == 3 ? u - qy * df : u;
                                const int tap = qs * nrt + u;
                                for (int h = 0; h < NH; ++h) {
                                    const int j = 4 * h + ln.kk;
                                    const int ao = bs_a_ofs(L, tl, NB, taps, ci, tap,
                                                            src_blade(NB, ln.i_a, j));
                                    const int64_t want_a =
                                        ((int64_t)(ci * L.Cout + tl.co_r) * taps + tap) * NB +
                                        src_blade(NB, ln.i_a, j);
                                    if (ao != want_a || ao < 0 || ao >= w_area)
                                        fail("block_small block %lld layer %d: A read at filter "
                                             "float %d, needs %lld", (long long)bid, li + 1, ao,
                                             (long long)want_a);
                                    const int bo = bs_b_ofs(L, tl, NB, ci, qs, qy, qx, h);
                                    if (bo < 0 || bo >= in_area) {
                                        fail("block_small block %lld layer %d: B read at float "
                                             "%d of %d", (long long)bid, li + 1, bo, in_area);
                                        continue;
                                    }
                                    // the element the product needs
                                    const int sl = tl.so + qs, yy = tl.yy + qy, xx = tl.xx + qx;
                                    if (li == 0) {
                                        const int64_t want =
                                            (((((int64_t)g.b * a.C0 + ci) * a.D0 + g.s0 + sl) *
                                                  (KD == 3 ? a.D0 : 1) + (KD == 3 ? yy : 0)) *
                                                 a.D0 + xx) * NB + j;
                                        if (band_src[(size_t)bo] != want)
                                            fail("block_small block %lld layer 1: B word %d holds "
                                                 "input float %lld, needs %lld", (long long)bid,
                                                 bo, (long long)band_src[(size_t)bo],
                                                 (long long)want);
                                    } else {
                                        const int want =
                                            ((ci * g.R1 + sl) * g.S1 + (KD == 3 ? yy * a.D1 : 0) +
                                             xx) * NB + j;
                                        if (bo != want || !y1_set[(size_t)bo])
                                            fail("block_small block %lld layer 2: B word %d (%s), "
                                                 "needs %d", (long long)bid, bo,
                                                 y1_set[(size_t)bo] ? "stored" : "never stored",
                                                 want);
                                    }
                                    if (current->errors >= 8) return;
                                }
                            }
                    // epilogue parameters (clamped channel; absent ones read input[0..3])
                    const int co_c = tl.co < L.Cout - 1 ? tl.co : L.Cout - 1;
                    if (bias && (int64_t)co_c * NB + ln.i0 + 4 > n_bias)
                        fail("block_small block %lld layer %d: bias read past the bias",
                             (long long)bid, li + 1);
                    if (act.mode == CLIFF_AGG_LINEAR &&
                        ((int64_t)co_c * act.K + act.K > buf_n(act.weight) ||
                         co_c >= buf_n(act.bias)))
                        fail("block_small block %lld layer %d: gate parameters past their "
                             "tensors", (long long)bid, li + 1);
                    // stores
                    if (tl.co >= L.Cout || tl.m >= npos) continue;
                    if (li == 0) {
                        const int o = bs_y1_ofs(g, NB, tl.co, tl.m, ln.i0);
                        const int want = (tl.co * g.R1 * g.S1 + tl.m) * NB + ln.i0;
                        if (o != want || o < 0 || o + 4 > y1_f) {
                            fail("block_small block %lld: intermediate store at %d, needs %d",
                                 (long long)bid, o, want);
                            continue;
                        }
                        for (int q = 0; q < 4; ++q) {
                            if (y1_set[(size_t)o + q])
                                fail("block_small block %lld: intermediate float %d stored twice",
                                     (long long)bid, o + q);
                            y1_set[(size_t)o + q] = 1;
                        }
                    } else {
                        const int64_t o = bs_y_ofs(a, g, NB, tl.co, tl.m, ln.i0);
                        const int sl = tl.m / g.S2, r = tl.m - sl * g.S2;
                        const int64_t want =
                            ((((int64_t)g.b * a.C2 + tl.co) * a.D2 + g.s0 + sl) * g.S2 + r) * NB +
                            ln.i0;
                        if (o != want || o < 0 || o + 4 > n_y || (o & 3)) {
                            fail("block_small block %lld: output store at %lld, needs %lld",
                                 (long long)bid, (long long)o, (long long)want);
                            continue;
                        }
                        uint8_t& w = written[(size_t)(o / 4)];
                        if (w) fail("block_small: output float %lld stored twice", (long long)o);
                        w = 1;
                    }
                }
                if (current->errors >= 8) return;
            }
            // layer 1 fills the whole intermediate band the second layer reads
            if (li == 0)
                for (int o = 0; o < a.C1 * g.R1 * g.S1 * NB; ++o)
                    if (!y1_set[(size_t)o]) {
                        fail("block_small block %lld: intermediate float %d never stored",
                             (long long)bid, o);
                        break;
                    }
        }
        current->workgroups++;
    }
    for (size_t i = 0; wstride == 1 && i < written.size(); ++i)
        if (!written[i]) {
            fail("block_small: output float %lld never stored", (long long)(i * 4));
            break;
        }
}

}  // namespace hostcheck
