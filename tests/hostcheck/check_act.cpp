// Host-side walk of act_kernel's address arithmetic (test infrastructure;
// see check_main.cpp), calling the kernel's own functions from act_geom.hpp:
// every thread's loads and stores inside the input and output, at the
// multivector of its (b, c) row and position, every output multivector
// written exactly once over the grid (all workgroups on grids of at most
// 2^15, else a sample, without the coverage count), and the gate's
// parameters inside their tensors.
#include <stdio.h>

#include <vector>

#include "act_geom.hpp"
#include "check.hpp"

namespace hostcheck {

using namespace cliff;

void check_act(const LaunchPlan& p)
{
    const ActKArgs& a = *static_cast<const ActKArgs*>(p.args);
    const int NB = p.tpl[0];
    const Buffer* bx = find_buffer(a.x);
    const Buffer* by = find_buffer(a.y);
    if (!bx || !by) {
        fail("act: a tensor pointer is not a case buffer");
        return;
    }
    if (p.block != ACT_THREADS || p.lds_bytes != 0 || (NB != 2 && NB != 4 && NB != 8))
        fail("act: workgroup %lld, LDS %lld, N_B %d", (long long)p.block, (long long)p.lds_bytes,
             NB);
    const int64_t rows = bx->n / (a.P * NB);
    if (rows * a.P * NB != bx->n || by->n != bx->n || rows % a.C ||
        p.grid != rows * a.n_pblk || a.n_pblk * ACT_THREADS * ACT_VPT < a.P ||
        (a.n_pblk - 1) * ACT_THREADS * ACT_VPT >= a.P)
        fail("act: grid %lld of %lld workgroups per row against %lld floats", (long long)p.grid,
             (long long)a.n_pblk, (long long)bx->n);
    if (a.act.mode == CLIFF_AGG_LINEAR) {
        const Buffer* bw = find_buffer(a.act.weight);
        const Buffer* bb = find_buffer(a.act.bias);
        if (!bw || !bb || bw->n < (int64_t)a.C * a.act.K || bb->n < a.C)
            fail("act: gate parameters smaller than [C, K] and [C]");
    }
    if (current->errors) return;
    const int64_t wstride = std::max<int64_t>(1, p.grid >> 15);
    current->grid_sampled |= wstride > 1;
    std::vector<uint8_t> written(wstride == 1 ? (size_t)(by->n / NB) : 0, 0);
    for (int64_t bid = 0; bid < p.grid; ++bid) {
        if (wstride > 1 && bid % wstride && bid >= 64 && bid < p.grid - 64) continue;
        const int64_t bc = act_bc(a, bid);
        if (bc < 0 || bc >= rows) {
            fail("act block %lld: row %lld of %lld", (long long)bid, (long long)bc,
                 (long long)rows);
            continue;
        }
        const int64_t base = act_base(a, bc, NB);
        for (int tid = 0; tid < ACT_THREADS; ++tid)
            for (int v = 0; v < ACT_VPT; ++v) {
                const int64_t pos = act_pos(a, bid, bc, tid, v);
                if (pos < 0) fail("act block %lld thread %d: position %lld", (long long)bid, tid,
                                  (long long)pos);
                if (pos < 0 || pos >= a.P) continue;  // not loaded, not stored
                const int64_t o = base + pos * NB;
                if (o != (bc * a.P + pos) * NB || o + NB > bx->n || o % (NB == 2 ? 2 : 4)) {
                    fail("act block %lld thread %d: multivector at float %lld", (long long)bid,
                         tid, (long long)o);
                    continue;
                }
                if (wstride == 1) {
                    if (written[(size_t)(o / NB)])
                        fail("act: multivector %lld written twice", (long long)(o / NB));
                    written[(size_t)(o / NB)] = 1;
                }
            }
        if (current->errors >= 8) return;
        current->workgroups++;
    }
    for (size_t i = 0; i < written.size(); ++i)
        if (!written[i]) {
            fail("act: multivector %lld never written", (long long)i);
            break;
        }
}

}  // namespace hostcheck
