// Device helpers for the multivector activation (paper, Algorithm 3), shared
// by the fused convolution epilogues and the standalone activation kernel.
#pragma once

#include "common.hpp"

namespace cliff {

// Position of blade `blade` in the gate's blade list, or -1 (a lookup in
// the table the host fills; for a blade known at compile time one argument
// word, else a chain of selects).
__device__ inline int gate_slot(const ActParams& act, int blade)
{
    int slot = act.slot[0];
#pragma unroll
    for (int b = 1; b < 8; ++b) slot = blade == b ? act.slot[b] : slot;
    return slot;
}

// Gate weight of `blade` for channel c: Linear -> weight[c, slot], Sum/Mean
// -> 1 for the selected blades; 0 for blades outside the subset.
__device__ inline float gate_coef(const ActParams& act, int slot, int c)
{
    if (slot < 0) return 0.0f;
    return act.mode == CLIFF_AGG_LINEAR ? act.weight[(int64_t)c * act.K + slot]
                                        : 1.0f;
}

// Gate value s from the full aggregated sum (Linear adds the channel's bias
// `lin_bias`, Mean divides by K), then sigmoid(s) = 1 / (1 + exp(-s)).
__device__ inline float gate_from_sum(const ActParams& act, float sum, float lin_bias)
{
    float s = sum;
    if (act.mode == CLIFF_AGG_LINEAR)
        s = s + lin_bias;
    else if (act.mode == CLIFF_AGG_MEAN)
        s = s / (float)act.K;
    return 1.0f / (1.0f + __expf(-s));
}

// The same for channel c, its Linear bias read from the descriptor.
__device__ inline float gate_sigmoid(const ActParams& act, float sum, int c)
{
    return gate_from_sum(act, sum, act.mode == CLIFF_AGG_LINEAR ? act.bias[c] : 0.0f);
}

}  // namespace cliff
