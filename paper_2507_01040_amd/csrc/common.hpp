// Shared definitions of the HIP kernels and the host dispatch code.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <initializer_list>

#include "cliffconv.h"

namespace cliff {

// Blade storage order is grade-then-lexicographic; inside the kernels a blade
// is handled as a bitmask over the generators (bit t-1 set <=> e_t present).
// The two orders differ only for k = 3, where slot 3 holds e3 (mask 4) and
// slot 4 holds e12 (mask 3); the map is its own inverse.
__host__ __device__ constexpr int blade_perm(int nb, int v)
{
    return nb == 8 ? (v == 3 ? 4 : (v == 4 ? 3 : v)) : v;
}

// For output blade i and input blade j (storage order), the filter blade whose
// product with e_j lands on e_i: e_src e_j = +-e_i, src = i XOR j on bitmasks.
__host__ __device__ constexpr int src_blade(int nb, int i, int j)
{
    return blade_perm(nb, blade_perm(nb, i) ^ blade_perm(nb, j));
}

// Signs of the table, bit e = i * nb + j: neg set => -1, zero set => 0,
// neither => +1.
struct SignMasks {
    uint64_t neg;
    uint64_t zero;
};

__host__ __device__ inline float sign_of(const SignMasks& s, int e)
{
    if ((s.zero >> e) & 1ull) return 0.0f;
    return ((s.neg >> e) & 1ull) ? -1.0f : 1.0f;
}

// Clears the calling thread's last HIP error before a launch, so that the
// status read after it (hipGetLastError) is the launch's own and not that of
// an earlier, unchecked call of the caller.
inline void clear_hip_error() { (void)hipGetLastError(); }

struct ActParams {
    int mode;     // -1: no activation
    int K;
    int slot[8];  // blade b's place in the gate's blade list, -1 if not in it
    const float* weight;
    const float* bias;
};

struct ConvProblem {
    int k, nb;
    int64_t B, C_in, C_out, d_image, d_filter, d_out;
    const float* x;
    const float* w;
    const float* bias;
    float* y;
    SignMasks sign;
    ActParams act;
    int mfma_shape;  // -1: chosen from the problem; 0..3: wide, medium, narrow, tiny
    int rowblk = 0;  // 2D row-aligned blocks: 2 where they leave <= 2 % idle (wide tiles), 1 also where whole-row slabs do not fit
    int64_t* blocks_out = nullptr;  // set: the matrix-core tile only plans, stores its workgroup count here and launches nothing
};

// Two-layer block (conv + bias + act, twice) for the fused small-block kernel.
struct BlockProblem {
    int k;
    int64_t B, C_in, C_mid, C_out, d_image, d_filter;
    const float* x;
    const float* w1;
    const float* b1;
    const float* w2;
    const float* b2;
    float* y;
    SignMasks sign;
    ActParams act1, act2;
};

// Launch logging: with the environment variable CLIFFCONV_DEBUG set to a
// non-zero value, every launch prints its kernel, grid and tiling to stderr.
bool debug_enabled();

// Compute units of the current device (cached per device); 0 on error.  With
// a launch observer installed: the observer's count.
int device_cus();

// Launch observation, for the host-side bounds checker (test
// infrastructure): a CPU build of the library installs an observer, and every
// launcher then hands it the launch's plan (kernel, template arguments, grid,
// workgroup size, LDS bytes, argument block) instead of enqueueing the
// kernel, and returns CLIFF_OK.  The checker walks the kernel's address
// arithmetic over every workgroup and lane of the plan.  No observer is ever
// installed in the library built for the GPU.
enum LaunchKind {
    LAUNCH_CONV_MFMA = 1,
    LAUNCH_CONV1D_MFMA,
    LAUNCH_CONV_DIRECT,
    LAUNCH_LINEAR_MFMA,
    LAUNCH_BLOCK_SMALL,
    LAUNCH_ACT,
};
struct LaunchPlan {
    int kind;
    int tpl[12];  // the kernel's template arguments, in declaration order
    int64_t grid, block, lds_bytes;
    const void* args;  // the kernel's argument block
};
struct LaunchObserver {
    int cus;  // compute units the dispatch heuristics assume
    void (*on_launch)(const LaunchPlan& plan, void* ctx);
    void* ctx;
};
extern LaunchObserver* launch_observer;

// Hands the plan to the observer if one is installed (then the caller does
// not launch).
inline bool observe_launch(int kind, std::initializer_list<int> tpl, int64_t grid,
                           int64_t block, int64_t lds_bytes, const void* args)
{
    if (!launch_observer) return false;
    LaunchPlan p;
    p.kind = kind;
    int n = 0;
    for (int v : tpl) p.tpl[n < 12 ? n++ : 11] = v;
    for (; n < 12; ++n) p.tpl[n] = 0;
    p.grid = grid;
    p.block = block;
    p.lds_bytes = lds_bytes;
    p.args = args;
    launch_observer->on_launch(p, launch_observer->ctx);
    return true;
}

// host-side launchers (defined in the .hip files)
cliff_status launch_conv_direct(const ConvProblem& p, hipStream_t stream);
// Returns CLIFF_EUNSUPPORTED without launching when no MFMA tiling fits.
cliff_status launch_conv_mfma(const ConvProblem& p, hipStream_t stream);
// k = 1 on the matrix cores; CLIFF_EUNSUPPORTED without launching likewise.
cliff_status launch_conv1d_mfma(const ConvProblem& p, hipStream_t stream);
// Linear layers (d_image = d_filter = 1) on the streamed MFMA kernel;
// CLIFF_EUNSUPPORTED without launching when the channel counts do not fit it.
cliff_status launch_linear_mfma(const ConvProblem& p, hipStream_t stream);
// The fused small-block kernel; CLIFF_EUNSUPPORTED without launching when its
// LDS working set does not fit.
cliff_status launch_block_small(const BlockProblem& p, hipStream_t stream);
int64_t block_small_lds_bytes(int k, int64_t C0, int64_t C1, int64_t C2, int64_t d_image,
                              int64_t d_filter, int64_t R);
cliff_status launch_act(int nb, int64_t B, int64_t C, int64_t P,
                        const ActParams& a, const float* x, float* y,
                        hipStream_t stream);

}  // namespace cliff
