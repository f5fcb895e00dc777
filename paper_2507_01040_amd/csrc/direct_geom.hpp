// Address arithmetic of conv_direct_kernel (one thread per output
// multivector), shared with the host-side bounds checker (a CPU build of the
// library used by the tests): the thread's (batch entry, output channel,
// position) and the input, filter and output offsets it reads and writes.
#pragma once

#include <stdint.h>

#include "common.hpp"

namespace cliff {

struct DirectArgs {
    const float* x;
    const float* w;
    const float* bias;
    float* y;
    int64_t total;  // B * C_out * d_out^k
    int C_in, C_out, D, Do, df;
    int64_t npos, nimg, ntap;  // d_out^k, d_image^k, d_filter^k
    SignMasks sign;
    ActParams act;
};

// Thread t (< total) computes output[b, co, position sp]; pbase is the flat
// input index of that position (tap 0): its coordinates read in base D.
struct DirectThread {
    int64_t b, sp, pbase;
    int co;
};

template <int KD>
__host__ __device__ inline DirectThread direct_thread(const DirectArgs& a, int64_t t)
{
    DirectThread d;
    d.sp = t % a.npos;
    const int64_t bc = t / a.npos;
    d.co = (int)(bc % a.C_out);
    d.b = bc / a.C_out;
    int pc[KD];
    int64_t r = d.sp;
    for (int k = KD - 1; k >= 0; --k) {
        pc[k] = (int)(r % a.Do);
        r /= a.Do;
    }
    d.pbase = 0;
    for (int k = 0; k < KD; ++k) d.pbase = d.pbase * a.D + pc[k];
    return d;
}

// Float offsets: input channel ci's multivector at the thread's position
// (plus direct_qoff for tap q), the filter [ci, co] taps, the output.
__host__ __device__ inline int64_t direct_x(const DirectArgs& a, const DirectThread& d, int ci,
                                            int NB)
{
    return ((d.b * a.C_in + ci) * a.nimg + d.pbase) * NB;
}
__host__ __device__ inline int64_t direct_w(const DirectArgs& a, const DirectThread& d, int ci,
                                            int NB)
{
    return ((int64_t)ci * a.C_out + d.co) * a.ntap * NB;
}
template <int KD>
__host__ __device__ inline int64_t direct_qoff(const DirectArgs& a, int64_t q)
{
    int64_t qoff = 0, r = q, scale = 1;
    for (int k = KD - 1; k >= 0; --k) {
        qoff += (r % a.df) * scale;
        r /= a.df;
        scale *= a.D;
    }
    return qoff;
}

}  // namespace cliff
