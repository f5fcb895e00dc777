/*
 * Measurement aid shipped with libcliffconv.so: not part of the layer API.
 *
 * The fp32 matrix-core peak that the chip actually sustains (clock under
 * load, issue limits) differs from the nominal 157.3 TFLOP/s (256 CUs x
 * 2.4 GHz x 256 FLOP/clock/CU).  The benchmark reports the convolution
 * kernels against both; this probe measures the sustained one.
 */
#ifndef CLIFFCONV_PROBE_H
#define CLIFFCONV_PROBE_H

#include <stdint.h>

#include "cliffconv.h"

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Enqueues one launch of n_workgroups workgroups of 256 threads; each wave
 * issues iters x 16 independent v_mfma_f32_16x16x4_f32 (2048 FLOP each) from
 * registers, with no memory traffic in the loop, and finally writes one float
 * per thread to out (device, n_workgroups x 256 floats, caller-owned) so the
 * work cannot be removed.  FLOPs per launch = n_workgroups x 4 x iters x 16 x
 * 2048.  CLIFF_EINVAL for a NULL out; CLIFF_ESHAPE unless
 * 1 <= n_workgroups < 2^31 and 1 <= iters; CLIFF_EDEVICE on a launch error.
 */
cliff_status cliffconv_mfma_peak_probe(int64_t n_workgroups, int32_t iters, float* out,
                                       void* stream);

#ifdef __cplusplus
}
#endif

#endif /* CLIFFCONV_PROBE_H */
