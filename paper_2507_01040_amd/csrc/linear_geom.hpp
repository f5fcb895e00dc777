// Address arithmetic of linear_mfma_kernel (the streamed Clifford linear
// layer): the LDS layout of the resident weight and epilogue parameters,
// which LDS word each A fragment reads, which input floats each lane loads
// and where its stores go.  The kernel and the host-side bounds checker (a
// CPU build of the library used by the tests) both call these functions, so
// the checker verifies the kernel's own arithmetic.
#pragma once

#include <stdint.h>

#include "common.hpp"

namespace cliff {

struct LinArgs {
    const float* x;
    const float* w;
    const float* bias;
    float* y;
    int64_t B;     // positions (rows of X and Y)
    int64_t n_wt;  // wave tiles: ceil(B / (16 NWW))
    int C_in;
    int WP;        // LDS floats per input channel of the weight (N plus padding)
    SignMasks sign;
    ActParams act;
};

// LDS: the raw weight [C_in][N] in rows of WP floats (NEG: then its negation
// in the same layout), then the bias [N], each (channel, blade)'s gate
// coefficient [N] and each channel's gate bias [N / N_B].
__host__ __device__ inline int lin_wfloats(const LinArgs& a) { return a.C_in * a.WP; }
// float4 e of the weight tensor (e < C_in N / 4) lands at this LDS float
__host__ __device__ inline int lin_w_lds(const LinArgs& a, int N, int e)
{
    const int ci = e / (N / 4), c4 = e - ci * (N / 4);
    return ci * a.WP + c4 * 4;
}
__host__ __device__ inline int lin_tail(const LinArgs& a, bool neg)
{
    return (neg ? 2 : 1) * lin_wfloats(a);
}

// A fragment lane (row n of a row tile, K slot r): row = (co, i) with
// i = n % NB; step t of a chunk reads input channel (4 r + t) / NB of the
// chunk and blade j = (4 r + t) % NB, i.e. weight blade src(i, j) (in the
// negated copy where `neg`).  Step s of the tile (chunk s / 4, t = s % 4),
// row tile rt: LDS float lin_a_base(t) + lin_a_step(s, rt).
__host__ __device__ inline int lin_a_base(const LinArgs& a, int NB, int n, int r, int t, bool neg)
{
    const int i = n % NB;
    const int k0 = 4 * r + t, ci0 = k0 / NB, j = k0 % NB;
    return ci0 * a.WP + (n - i) + src_blade(NB, i, j) + (neg ? lin_wfloats(a) : 0);
}
__host__ __device__ inline int lin_a_step(const LinArgs& a, int NB, int s, int rt)
{
    return (s / 4) * ((16 / NB) * a.WP) + 16 * rt;
}

// Input: lane (n, r) of column tile nw of wave tile tt loads row m = tt TP +
// nw 16 + n (past B: the last row, loaded but never stored), floats 4 r ..
// 4 r + 3 of each chunk of 16: input float lin_x_row(...) + 16 chunk.
__host__ __device__ inline int64_t lin_x_row(const LinArgs& a, int K, int TP, int64_t tt, int nw,
                                             int n, int r)
{
    const int64_t m = tt * TP + nw * 16 + n;
    return (m < a.B ? m : a.B - 1) * K + 4 * r;
}

// Output: wave tile tt's rows m0 = tt TP .. m0 + lin_y_rows - 1 go through a
// buffer descriptor of that many rows (the hardware drops stores past it);
// lane (n, r) stores its D fragment of row tile rt, column tile nw (columns
// row0 .. row0 + 3, row0 = 16 rt + 4 r) at byte lin_y_byte from row m0.
__host__ __device__ inline int64_t lin_y_rows(const LinArgs& a, int TP, int64_t tt)
{
    const int64_t m0 = tt * TP;
    return a.B - m0 < TP ? a.B - m0 : TP;
}
__host__ __device__ inline int lin_y_byte(int N, int nw, int n, int row0)
{
    return ((nw * 16 + n) * N + row0) * 4;
}

}  // namespace cliff
