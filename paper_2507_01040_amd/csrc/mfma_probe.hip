// Sustained fp32 matrix-core throughput: every wave issues independent
// v_mfma_f32_16x16x4_f32 from registers, with no memory traffic in the loop.
// Each wave keeps 16 accumulator chains: measured, 8 chains per wave reach
// only ~90 % of the pipe even with several waves per SIMD, 16 reach ~99 %.
#include "cliffconv_probe.h"
#include "common.hpp"

namespace cliff {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void mfma_peak_kernel(int iters, float* out)
{
    f4 acc[16];
#pragma unroll
    for (int t = 0; t < 16; ++t) acc[t] = f4{0.f, 0.f, 0.f, 0.f};
    const float a = 1e-3f * (float)threadIdx.x;
    const float b = 1e-3f * (float)blockIdx.x;
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int t = 0; t < 16; ++t)
            acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc[t], 0, 0, 0);
    }
    float s = 0.f;
#pragma unroll
    for (int t = 0; t < 16; ++t) s += acc[t][0] + acc[t][1] + acc[t][2] + acc[t][3];
    out[(int64_t)blockIdx.x * 256 + threadIdx.x] = s;
}

}  // namespace
}  // namespace cliff

extern "C" cliff_status cliffconv_mfma_peak_probe(int64_t n_workgroups, int32_t iters,
                                                  float* out, void* stream)
{
    if (!out) return CLIFF_EINVAL;
    if (n_workgroups < 1 || n_workgroups >= (1ll << 31) || iters < 1) return CLIFF_ESHAPE;
    cliff::clear_hip_error();
    hipLaunchKernelGGL(cliff::mfma_peak_kernel, dim3((unsigned)n_workgroups), dim3(256), 0,
                       (hipStream_t)stream, (int)iters, out);
    return hipGetLastError() == hipSuccess ? CLIFF_OK : CLIFF_EDEVICE;
}
