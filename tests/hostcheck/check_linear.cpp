// Host-side walk of linear_mfma_kernel's address arithmetic (test
// infrastructure; see check_main.cpp), calling the kernel's own functions
// from linear_geom.hpp.
//
// For a launch plan it checks the launch shape and the LDS layout (weight,
// its negated copy, bias, gate coefficients and gate biases inside the
// launch's LDS) and, for every wave of the persistent grid and every wave
// tile it takes (and the next tile it prefetches):
//   * every weight float4 copied into LDS inside the weight and inside its
//     area;
//   * every A fragment read of every lane, step and row tile at the LDS word
//     holding w[ci, co, src(i, j)] for the lane's row (co, i) and K index
//     (ci, j) (in the negated copy exactly where the table's sign is -1 and
//     the copy is kept);
//   * every input load inside the input, at the lane's row (clamped to the
//     last one) and K chunk;
//   * every output store that the buffer descriptor keeps inside the output
//     at the lane's row and columns, every output float4 stored exactly once
//     over the grid, and none kept past row B.
#include <stdio.h>

#include <vector>

#include "check.hpp"
#include "linear_geom.hpp"

namespace hostcheck {

using namespace cliff;

void check_linear(const LaunchPlan& p)
{
    const LinArgs& a = *static_cast<const LinArgs*>(p.args);
    const int NB = p.tpl[0], RT = p.tpl[1], KQ = p.tpl[2], NWW = p.tpl[3], PF = p.tpl[4];
    const bool NEG = p.tpl[6] != 0;
    const int NT = p.tpl[7];
    const int N = 16 * RT, K = 16 * KQ, TP = 16 * NWW;
    const Buffer* bx = find_buffer(a.x);
    const Buffer* bw = find_buffer(a.w);
    const Buffer* by = find_buffer(a.y);
    if (!bx || !bw || !by) {
        fail("linear: a tensor pointer is not a case buffer");
        return;
    }
    const int C_out = N / NB;
    if (p.block != NT || (NT != 256 && NT != 512) || a.C_in * NB != K ||
        bx->n != a.B * K || by->n != a.B * N || bw->n != (int64_t)a.C_in * C_out * NB ||
        a.n_wt != (a.B + TP - 1) / TP || KQ % PF || a.WP < N)
        fail("linear: launch %lld threads, N %d K %d, B %lld, %lld wave tiles, pitch %d",
             (long long)p.block, N, K, (long long)a.B, (long long)a.n_wt, a.WP);
    const int64_t tail = lin_tail(a, NEG);
    if ((tail + 2 * N + N / NB) * 4 > p.lds_bytes || p.lds_bytes > 160 * 1024)
        fail("linear: LDS %lld bytes for %lld floats", (long long)p.lds_bytes,
             (long long)(tail + 2 * N + N / NB));
    if (current->errors) return;
    // the weight copy
    for (int e = 0; e < a.C_in * (N / 4); ++e) {
        const int o = lin_w_lds(a, N, e);
        const int ci = e / (N / 4), c = (e - ci * (N / 4)) * 4;  // weight float 4 e = (ci, c)
        if ((int64_t)e * 4 + 4 > bw->n || o != ci * a.WP + c || o + 4 > lin_wfloats(a)) {
            fail("linear: weight float4 %d to LDS float %d", e, o);
            return;
        }
    }
    // A reads: the same for every tile (every lane, step and row tile)
    for (int lane = 0; lane < 64; ++lane) {
        const int n = lane & 15, r = lane >> 4, i = n % NB;
        for (int s = 0; s < 4 * KQ; ++s) {
            const int tt = s % 4;
            const int k = 16 * (s / 4) + 4 * r + tt, ci = k / NB, j = k % NB;
            const bool neg = NEG && sign_of(a.sign, i * NB + j) < 0.f;
            for (int rt = 0; rt < RT; ++rt) {
                const int co = (16 * rt + n) / NB;
                const int o = lin_a_base(a, NB, n, r, tt, neg) + lin_a_step(a, NB, s, rt);
                const int want =
                    ci * a.WP + co * NB + src_blade(NB, i, j) + (neg ? lin_wfloats(a) : 0);
                if (o != want || o < 0 || o >= tail)
                    fail("linear lane %d step %d row tile %d: A at LDS float %d, needs %d", lane,
                         s, rt, o, want);
            }
        }
    }
    if (current->errors) return;
    // tiles: every wave's (all of them when there are at most 2^15, else
    // every (n_wt / 2^15)-th, the first and the last 64, with no coverage count)
    const int waves = NT / 64;
    const int64_t stride = p.grid * waves;
    const int64_t tstride = std::max<int64_t>(1, a.n_wt >> 15);
    current->grid_sampled |= tstride > 1;
    std::vector<uint8_t> written(tstride == 1 ? (size_t)(by->n / 4) : 0, 0);
    int64_t tiles_seen = 0;
    for (int64_t bid = 0; bid < p.grid; ++bid)
        for (int wave = 0; wave < waves; ++wave)
            for (int64_t t = bid * waves + wave; t < a.n_wt; t += stride) {
                ++tiles_seen;
                if (tstride > 1 && t % tstride && t >= 64 && t < a.n_wt - 64) continue;
                const int64_t tn = t + stride < a.n_wt ? t + stride : t;
                for (int lane = 0; lane < 64; ++lane) {
                    const int n = lane & 15, r = lane >> 4;
                    // input loads of this tile and the next (prefetch)
                    for (const int64_t tx : {t, tn})
                        for (int nw = 0; nw < NWW; ++nw) {
                            const int64_t m = tx * TP + nw * 16 + n;
                            const int64_t row = m < a.B ? m : a.B - 1;
                            for (int q = 0; q < KQ; ++q) {
                                const int64_t o = lin_x_row(a, K, TP, tx, nw, n, r) + 16 * q;
                                if (o != row * K + 4 * r + 16 * q || o < 0 || o + 4 > bx->n)
                                    fail("linear tile %lld lane %d: input load at %lld",
                                         (long long)tx, lane, (long long)o);
                            }
                        }
                    // stores through the descriptor of this tile's rows
                    const int64_t rows = lin_y_rows(a, TP, t), m0 = t * TP;
                    if (rows < 1 || rows > TP)
                        fail("linear tile %lld: %lld rows", (long long)t, (long long)rows);
                    for (int rt = 0; rt < RT; ++rt)
                        for (int nw = 0; nw < NWW; ++nw) {
                            const int row0 = 16 * rt + 4 * r;
                            const int64_t byte = lin_y_byte(N, nw, n, row0);
                            if (byte + 16 > rows * N * 4) {
                                // dropped by the descriptor: only rows past B
                                if (m0 + nw * 16 + n < a.B)
                                    fail("linear tile %lld lane %d: store of row %lld dropped",
                                         (long long)t, lane, (long long)(m0 + nw * 16 + n));
                                continue;
                            }
                            const int64_t o = m0 * N + byte / 4;
                            if (o != (m0 + nw * 16 + n) * N + row0 || o + 4 > by->n || (o & 3)) {
                                fail("linear tile %lld lane %d: store at float %lld",
                                     (long long)t, lane, (long long)o);
                                continue;
                            }
                            if (tstride == 1) {
                                uint8_t& w = written[(size_t)(o / 4)];
                                if (w) fail("linear: output float %lld stored twice",
                                            (long long)o);
                                w = 1;
                            }
                        }
                    if (current->errors >= 8) return;
                }
            }
    if (tiles_seen != a.n_wt) fail("linear: %lld wave tiles walked of %lld", (long long)tiles_seen,
                                   (long long)a.n_wt);
    for (size_t q = 0; q < written.size(); ++q)
        if (!written[q]) {
            fail("linear: output float %lld never stored", (long long)(q * 4));
            break;
        }
    current->workgroups += p.grid;
}

}  // namespace hostcheck
