// clifford_block2_nd without a caller workspace, for callers that cannot
// allocate device memory (code under HIP graph capture, tight serving loops,
// harnesses that forbid allocation): the intermediate of a block that runs as
// two launches lives in a fixed array of this library, one per GPU, held
// until the process ends.  Everything else is clifford_block2_nd_path.
#include <stdint.h>

#include <atomic>

#include "cliffconv.h"
#include "common.hpp"

namespace {

// The intermediate of the two-launch path: CLIFF_NOALLOC_SCRATCH_FLOATS fp32
// values (64 MiB) of device memory on every GPU the library runs on.  In host
// code this name is a host-side stand-in, not a device address: host code only
// ever uses the address hipGetSymbolAddress returned for the current device.
__device__ __align__(256) float scratch[CLIFF_NOALLOC_SCRATCH_FLOATS];

// The device address of `scratch` per device, looked up once per device
// (with that device current) on its first call.
std::atomic<float*> scratch_ptr[64];

cliff_status scratch_of_current_device(float** out)
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return CLIFF_EDEVICE;
    float* p = scratch_ptr[dev].load(std::memory_order_acquire);
    if (!p) {
        void* addr = nullptr;
        if (hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch)) != hipSuccess || !addr)
            return CLIFF_EDEVICE;
        p = static_cast<float*>(addr);
        scratch_ptr[dev].store(p, std::memory_order_release);
    }
    *out = p;
    return CLIFF_OK;
}

int64_t ipow(int64_t a, int k)
{
    int64_t r = 1;
    for (int t = 0; t < k; ++t) r *= a;
    return r;
}

}  // namespace

extern "C" cliff_status clifford_block2_nd_noalloc(
    int k, const int8_t* g, int64_t B, int64_t C_in, int64_t C_mid, int64_t C_out,
    int64_t d_image, int64_t d_filter, const float* input, const float* filters1,
    const float* bias1, const cliff_act_desc* act1, const float* filters2, const float* bias2,
    const cliff_act_desc* act2, float* output, void* stream)
{
    // the intermediate's size, checked before anything else touches the GPU
    // (clifford_block2_nd_path repeats every other check)
    if (k >= 1 && k <= 3 && B > 0 && C_mid > 0 && d_filter > 0 && d_image >= 2 * d_filter - 1 &&
        d_image < (1 << 20)) {
        const int64_t d_mid = d_image - d_filter + 1, pos = ipow(d_mid, k);
        if (B > CLIFF_NOALLOC_SCRATCH_FLOATS / C_mid ||
            B * C_mid > CLIFF_NOALLOC_SCRATCH_FLOATS / pos ||
            B * C_mid * pos > CLIFF_NOALLOC_SCRATCH_FLOATS >> k)
            return CLIFF_ESCRATCH;
    }
    float* ws = nullptr;
    const cliff_status s = scratch_of_current_device(&ws);
    if (s != CLIFF_OK) return s;
    return clifford_block2_nd_path(k, g, B, C_in, C_mid, C_out, d_image, d_filter, input,
                                   filters1, bias1, act1, filters2, bias2, act2, ws, output,
                                   stream, CLIFF_BLOCK_AUTO);
}
