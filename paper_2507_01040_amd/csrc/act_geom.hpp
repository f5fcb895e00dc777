// Address arithmetic of act_kernel (the standalone multivector activation),
// shared with the host-side bounds checker (a CPU build of the library used
// by the tests): which (batch entry, channel) row and positions a thread
// handles, and where they are.
#pragma once

#include <stdint.h>

#include "common.hpp"

namespace cliff {

constexpr int ACT_THREADS = 256;
constexpr int ACT_VPT = 2;  // multivectors per thread (measured: 2 is best or tied at 0.27-1.3 GB)

struct ActKArgs {
    const float* x;
    float* y;
    int64_t P;       // positions per (b, c)
    int64_t n_pblk;  // workgroups per (b, c)
    int C;
    ActParams act;
};

// Workgroup bid works on row bc = b * C + c of [B, C, P, N_B], positions
// act_pos(v) for v < ACT_VPT of each thread (those below P).
__host__ __device__ inline int64_t act_bc(const ActKArgs& a, int64_t bid) { return bid / a.n_pblk; }
__host__ __device__ inline int64_t act_base(const ActKArgs& a, int64_t bc, int NB)
{
    return bc * a.P * NB;
}
__host__ __device__ inline int64_t act_pos(const ActKArgs& a, int64_t bid, int64_t bc, int tid,
                                           int v)
{
    return (bid - bc * a.n_pblk) * (ACT_THREADS * ACT_VPT) + tid + v * ACT_THREADS;
}

}  // namespace cliff
