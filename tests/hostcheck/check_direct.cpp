// Host-side walk of conv_direct_kernel's address arithmetic (test
// infrastructure; see check_main.cpp), calling the kernel's own functions
// from direct_geom.hpp: for every thread (all of them on grids of at most
// 2^15 workgroups, else a sample), every input read at input[b, ci, p + q, j]
// for the thread's position p, every filter read at filters[ci, co, q, .],
// the bias and gate parameters inside their tensors, and the output
// multivector stored at its own place, each once over the grid.
#include <stdio.h>

#include <vector>

#include "check.hpp"
#include "direct_geom.hpp"

namespace hostcheck {

using namespace cliff;

namespace {

template <int KD>
void walk(const LaunchPlan& p, const DirectArgs& a, int NB, const Buffer* bx, const Buffer* bw,
          const Buffer* by)
{
    const int64_t gstride = std::max<int64_t>(1, p.grid >> 15);
    current->grid_sampled |= gstride > 1;
    std::vector<uint8_t> written(gstride == 1 ? (size_t)(by->n / NB) : 0, 0);
    for (int64_t bid = 0; bid < p.grid; ++bid) {
        if (gstride > 1 && bid % gstride && bid >= 64 && bid < p.grid - 64) continue;
        for (int tid = 0; tid < 256; ++tid) {
            const int64_t t = bid * 256 + tid;
            if (t >= a.total) break;  // the kernel returns
            const DirectThread d = direct_thread<KD>(a, t);
            // the thread's position coordinates, most significant first
            int64_t c[3] = {0, 0, 0}, r = d.sp;
            for (int k = KD - 1; k >= 0; --k) {
                c[k] = r % a.Do;
                r /= a.Do;
            }
            if (d.b < 0 || d.co < 0 || d.co >= a.C_out || d.b * a.C_out * a.npos + d.co * a.npos +
                                                              d.sp != t)
                fail("direct thread %lld: b %lld co %d position %lld", (long long)t,
                     (long long)d.b, d.co, (long long)d.sp);
            // the first and last input channels bound all (offsets grow with ci)
            for (int ci : {0, a.C_in - 1})
                for (int64_t q = 0; q < a.ntap; ++q) {
                    int64_t qc[3] = {0, 0, 0}, rq = q;
                    for (int k = KD - 1; k >= 0; --k) {
                        qc[k] = rq % a.df;
                        rq /= a.df;
                    }
                    int64_t want = d.b * a.C_in + ci;
                    for (int k = 0; k < KD; ++k) want = want * a.D + c[k] + qc[k];
                    const int64_t xo = direct_x(a, d, ci, NB) + direct_qoff<KD>(a, q) * NB;
                    if (xo != want * NB || xo < 0 || xo + NB > bx->n)
                        fail("direct thread %lld: input at %lld, needs %lld", (long long)t,
                             (long long)xo, (long long)(want * NB));
                    const int64_t wo = direct_w(a, d, ci, NB) + q * NB;
                    if (wo != (((int64_t)ci * a.C_out + d.co) * a.ntap + q) * NB || wo < 0 ||
                        wo + NB > bw->n)
                        fail("direct thread %lld: filter at %lld", (long long)t, (long long)wo);
                    if (current->errors >= 8) return;
                }
            if (a.bias && (int64_t)d.co * NB + NB > find_buffer(a.bias)->n)
                fail("direct thread %lld: bias read past the bias", (long long)t);
            if (a.act.mode == CLIFF_AGG_LINEAR &&
                ((int64_t)d.co * a.act.K + a.act.K > find_buffer(a.act.weight)->n ||
                 d.co >= find_buffer(a.act.bias)->n))
                fail("direct thread %lld: gate parameters past their tensors", (long long)t);
            if ((t + 1) * NB > by->n) fail("direct thread %lld: output past the output", (long long)t);
            if (gstride == 1) {
                if (written[(size_t)t]) fail("direct: output %lld stored twice", (long long)t);
                written[(size_t)t] = 1;
            }
        }
        current->workgroups++;
    }
    for (size_t i = 0; i < written.size(); ++i)
        if (!written[i]) {
            fail("direct: output multivector %lld never stored", (long long)i);
            break;
        }
}

}  // namespace

void check_direct(const LaunchPlan& p)
{
    const DirectArgs& a = *static_cast<const DirectArgs*>(p.args);
    const int KD = p.tpl[0], NB = p.tpl[1];
    const Buffer* bx = find_buffer(a.x);
    const Buffer* bw = find_buffer(a.w);
    const Buffer* by = find_buffer(a.y);
    if (!bx || !bw || !by) {
        fail("direct: a tensor pointer is not a case buffer");
        return;
    }
    if (p.block != 256 || p.lds_bytes != 0 || p.grid != (a.total + 255) / 256 ||
        by->n != a.total * NB || NB != (1 << KD))
        fail("direct: grid %lld of 256 for %lld outputs", (long long)p.grid, (long long)a.total);
    if (current->errors) return;
    if (KD == 1) walk<1>(p, a, NB, bx, bw, by);
    if (KD == 2) walk<2>(p, a, NB, bx, bw, by);
    if (KD == 3) walk<3>(p, a, NB, bx, bw, by);
}

}  // namespace hostcheck
