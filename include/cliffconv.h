/*
 * cliffconv.h -- C ABI of the MI355X (gfx950) Clifford convolution library
 * (libcliffconv.so).
 *
 * The operations are those of "Fast Clifford Neural Layers" (arXiv
 * 2507.01040): the k-D Clifford convolution of Algorithm 1 and the Clifford
 * linear layer of Algorithm 2, each with the bias add, the multivector
 * activation of Algorithm 3, usable on its own or fused as their epilogue,
 * and the two-layer block (convolution + activation, twice) the paper builds
 * its networks from.  All arithmetic is IEEE fp32 on the GPU.
 *
 * Algebra (paper, Background, "Clifford Algebra"): Cl_g(R^k) with signature
 * g in {-1, 0, +1}^k, generators e_1..e_k, e_i e_i = g_i, e_i e_j = -e_j e_i.
 * A signature is valid if at least one g_i is non-zero.  A multivector holds
 * N_B = 2^k real blade coefficients, stored contiguously in this order
 * (grade first, then lexicographic):
 *     k = 1: (1, e1)
 *     k = 2: (1, e1, e2, e12)
 *     k = 3: (1, e1, e2, e3, e12, e13, e23, e123)
 * Blade indices in this API are 0-based.
 *
 * Common conventions
 *  - Every tensor is dense, row-major, fp32, with the blade index last.
 *    Spatial indices are row-major with the first spatial axis slowest.
 *  - Device pointers point to memory of the current HIP device.  The caller
 *    owns every buffer; the library never allocates or frees device memory in
 *    these calls and keeps no pointer after a call returns.
 *  - Calls enqueue work on `stream` (a hipStream_t passed as void*; NULL is
 *    the null stream) and return without synchronising.  Results are visible
 *    once the stream has reached the work.
 *  - Errors are returned, never raised: argument checks happen before any
 *    work is enqueued, and on an argument error the output is left untouched.
 *    CLIFF_EDEVICE reports a HIP launch error (hipGetLastError) after the
 *    launch; the output content is then undefined.
 *  - Thread safety: calls may be made concurrently from several host threads.
 *  - With the environment variable CLIFFCONV_DEBUG set (non-zero), every
 *    kernel launch prints its kernel, grid and tiling to stderr.
 */
#ifndef CLIFFCONV_H
#define CLIFFCONV_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    CLIFF_OK = 0,
    CLIFF_EINVAL = 1,       /* null pointer, bad k / signature / act descriptor */
    CLIFF_ESHAPE = 2,       /* non-positive size, d_filter > d_image, overflow */
    CLIFF_EALIGN = 3,       /* tensor pointer not 16-byte aligned */
    CLIFF_EOVERLAP = 4,     /* output memory overlaps an input */
    CLIFF_EUNSUPPORTED = 5, /* valid request the library does not support */
    CLIFF_EDEVICE = 6,      /* HIP reported an error */
    CLIFF_ESCRATCH = 7      /* intermediate larger than the library's fixed scratch
                               (clifford_block2_nd_noalloc only) */
} cliff_status;

/* Gate aggregation of Algorithm 3. */
typedef enum {
    CLIFF_AGG_LINEAR = 0, /* s = sum_t input[blade_idx[t]] * weight[c, t] + bias[c] */
    CLIFF_AGG_SUM = 1,    /* s = sum_t input[blade_idx[t]]                       */
    CLIFF_AGG_MEAN = 2    /* s = (sum_t input[blade_idx[t]]) / K                 */
} cliff_agg;

/*
 * Multivector activation descriptor (paper, Algorithm 3): for every
 * multivector of channel c the gate s is formed from the K selected blades
 * and every blade j is scaled, out[j] = in[j] * sigmoid(s), with
 * sigmoid(s) = 1 / (1 + exp(-s)).
 *   mode       cliff_agg
 *   K          number of gating blades, 1 <= K <= N_B
 *   blade_idx  K distinct 0-based blade indices (entries past K ignored);
 *              host memory, read during the call only
 *   weight     device [C, K] fp32, Linear only (ignored otherwise)
 *   bias       device [C] fp32, Linear only (ignored otherwise)
 * Spatial positions share the channel's weight and bias.
 */
typedef struct {
    int32_t mode;
    int32_t K;
    int32_t blade_idx[8];
    const float* weight;
    const float* bias;
} cliff_act_desc;

/*
 * k-D Clifford convolution (paper, Algorithm 1), no padding, unit stride, no
 * dilation, followed by the bias add and, if `act` is not NULL, the
 * multivector activation applied to the result:
 *
 *   output[b, co, p] = act( sum_{ci} sum_{q in [0, d_filter)^k}
 *                               filters[ci, co, q] * input[b, ci, p + q]
 *                           + bias[co] )
 *
 * where * is the geometric product with the filter on the left, and
 * p ranges over [0, d_out)^k with d_out = d_image - d_filter + 1.
 *
 *   k         1, 2 or 3 (N_B = 2^k), all on the matrix cores (shapes whose
 *             staging does not fit fall back to a per-output kernel).
 *   g         host int8[k], each in {-1, 0, +1}, not all 0
 *   input     device [B, C_in, d_image^k, N_B]
 *   filters   device [C_in, C_out, d_filter^k, N_B]
 *   bias      device [C_out, N_B], or NULL for zero
 *   output    device [B, C_out, d_out^k, N_B]; must not overlap any input
 *   act       NULL, or the activation to fuse (weight [C_out, K], bias [C_out])
 *   stream    hipStream_t or NULL
 * Alignment: input, filters, bias and output 16-byte aligned (CLIFF_EALIGN);
 * act->weight and act->bias 4-byte aligned.
 * Sizes: B, C_in, C_out, d_filter >= 1, d_image >= d_filter (CLIFF_ESHAPE);
 * every tensor must hold fewer than 2^40 elements.
 * B = 0 is accepted and enqueues nothing.
 */
cliff_status clifford_conv_nd(int k, const int8_t* g, int64_t B, int64_t C_in,
                              int64_t C_out, int64_t d_image, int64_t d_filter,
                              const float* input, const float* filters,
                              const float* bias, float* output,
                              const cliff_act_desc* act, void* stream);

/* Kernel choice for clifford_conv_nd_algo. */
typedef enum {
    CLIFF_ALGO_AUTO = 0,        /* what clifford_conv_nd does */
    CLIFF_ALGO_DIRECT = 1,      /* one thread per output multivector, fp32 FMA */
    CLIFF_ALGO_MFMA = 2,        /* implicit GEMM on fp32 MFMA, tile shape chosen
                                   from the problem size */
    CLIFF_ALGO_MFMA_WIDE = 3,   /* MFMA, forced tile shape, channels x
                                   positions per workgroup: k = 1: 64 x 128
                                   (d_filter = 17, layers of >= 1 GFLOP: 64
                                   x 176 where that fills the last round of
                                   compute units better); k = 2: 64 x 128,
                                   32 x 256 when C_out <= 32 or when a 64-
                                   channel stage does not fit, 16 x 512
                                   (C_out <= 16), 8 x 512 (C_out <= 8);
                                   k = 3: 16 x 128, with d_filter = 3 32 x
                                   128 (16 < C_out <= 32) and 8 x 256
                                   (C_out <= 8).  The automatic choice also
                                   takes the 96- and 112-position forms of
                                   the 64- (k = 2) and 32-channel (k = 3)
                                   tiles and the 384- and 256-position forms
                                   of the 16- and 8-channel ones on layers of
                                   >= 1 GFLOP, where they fill the last
                                   round of compute units better */
    CLIFF_ALGO_MFMA_MEDIUM = 4, /* MFMA, 64 / 64 / 32 (k=1/2/3) channels x 32
                                   positions */
    CLIFF_ALGO_MFMA_NARROW = 5, /* MFMA, 8 / 8 / 4 channels x 256 positions */
    CLIFF_ALGO_MFMA_TINY = 6,   /* MFMA, 8 / 4 / 2 channels x 32 positions
                                   (k = 2, 3: the K loop split over 4 waves) */
    CLIFF_ALGO_MFMA_STREAM = 7  /* MFMA, linear layers only (d_image =
                                   d_filter = 1, C_in N_B and C_out N_B each
                                   64, 128 or 256): persistent waves that
                                   stream 16-64 positions at a time past the
                                   weight held in LDS */
} cliff_algo;

/*
 * Same operation and contract as clifford_conv_nd, with the kernel family
 * (and for the MFMA family optionally the tile shape) forced;
 * CLIFF_EUNSUPPORTED if that choice cannot run the request.  For tests and
 * benchmarks that compare kernels.
 */
cliff_status clifford_conv_nd_algo(int k, const int8_t* g, int64_t B,
                                   int64_t C_in, int64_t C_out, int64_t d_image,
                                   int64_t d_filter, const float* input,
                                   const float* filters, const float* bias,
                                   float* output, const cliff_act_desc* act,
                                   void* stream, int algo);

/*
 * Clifford linear layer (paper, Algorithm 2), plus the bias add and, if
 * `act` is not NULL, the fused multivector activation:
 *
 *   output[b, co] = act( sum_{ci} weight[ci, co] * input[b, ci] + bias[co] )
 *
 * with the weight on the left of the geometric product.
 *   k, g      as for clifford_conv_nd
 *   input     device [B, C_in, N_B]
 *   weight    device [C_in, C_out, N_B]
 *   bias      device [C_out, N_B], or NULL for zero
 *   output    device [B, C_out, N_B]; must not overlap any input
 * Same alignment, size, error and stream rules as clifford_conv_nd; it is
 * the convolution with d_image = d_filter = 1.  Layers with C_in N_B and
 * C_out N_B each 64, 128 or 256 and B >= 16384 run on a streamed kernel that
 * keeps the weight in LDS (CLIFF_ALGO_MFMA_STREAM); other layers on the
 * convolution kernels.
 */
cliff_status clifford_linear(int k, const int8_t* g, int64_t B, int64_t C_in,
                             int64_t C_out, const float* input, const float* weight,
                             const float* bias, float* output,
                             const cliff_act_desc* act, void* stream);

/*
 * Two-layer Clifford block (the basic block pattern of the paper's
 * network-block experiments, Table 2): convolution (Algorithm 1) + bias +
 * optional activation (Algorithm 3), then a second convolution of the
 * intermediate + bias + optional activation:
 *
 *   mid    = act1( conv(input,  filters1) + bias1 )   [B, C_mid, d_mid^k, N_B]
 *   output = act2( conv(mid,    filters2) + bias2 )   [B, C_out, d_out^k, N_B]
 *
 * with d_mid = d_image - d_filter + 1 and d_out = d_mid - d_filter + 1 (both
 * layers share d_filter, no padding, unit stride).
 *   k, g               as for clifford_conv_nd (k = 1 runs as two launches)
 *   filters1, bias1    device [C_in, C_mid, d_filter^k, N_B], [C_mid, N_B] or NULL
 *   act1               NULL or the first activation (weight [C_mid, K], bias [C_mid])
 *   filters2, bias2    device [C_mid, C_out, d_filter^k, N_B], [C_out, N_B] or NULL
 *   act2               NULL or the second activation (weight [C_out, K], bias [C_out])
 *   workspace          device, caller-owned, B * C_mid * d_mid^k * N_B floats:
 *                      holds `mid` when the block runs as two launches; its
 *                      contents are unspecified afterwards
 *   output             device [B, C_out, d_out^k, N_B]
 * Small blocks (few channels, little work) run as one fused launch that keeps
 * `mid` in on-chip memory; others as two clifford_conv_nd launches through the
 * workspace.  Both give the same results up to fp32 rounding order.
 * Errors: as clifford_conv_nd (CLIFF_EINVAL also for a NULL workspace or
 * second filter; CLIFF_ESHAPE unless d_image >= 2 d_filter - 1); the
 * workspace and the output must not overlap each other or any input
 * (CLIFF_EOVERLAP).  16-byte alignment for all tensors.
 */
cliff_status clifford_block2_nd(int k, const int8_t* g, int64_t B, int64_t C_in,
                                int64_t C_mid, int64_t C_out, int64_t d_image,
                                int64_t d_filter, const float* input,
                                const float* filters1, const float* bias1,
                                const cliff_act_desc* act1, const float* filters2,
                                const float* bias2, const cliff_act_desc* act2,
                                float* workspace, float* output, void* stream);

/* Execution path for clifford_block2_nd_path. */
typedef enum {
    CLIFF_BLOCK_AUTO = 0,        /* what clifford_block2_nd does */
    CLIFF_BLOCK_TWO_LAUNCH = 1,  /* two clifford_conv_nd launches via the workspace */
    CLIFF_BLOCK_FUSED = 2        /* one fused launch (k = 2, 3); CLIFF_EUNSUPPORTED
                                    when its on-chip working set does not fit */
} cliff_block_path;

/* clifford_block2_nd with the execution path forced (tests, benchmarks). */
cliff_status clifford_block2_nd_path(int k, const int8_t* g, int64_t B, int64_t C_in,
                                     int64_t C_mid, int64_t C_out, int64_t d_image,
                                     int64_t d_filter, const float* input,
                                     const float* filters1, const float* bias1,
                                     const cliff_act_desc* act1, const float* filters2,
                                     const float* bias2, const cliff_act_desc* act2,
                                     float* workspace, float* output, void* stream,
                                     int path);

/*
 * clifford_block2_nd for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the same block, without the workspace argument.  A block that
 * runs as two launches keeps its intermediate in a fixed array inside the
 * library instead: CLIFF_NOALLOC_SCRATCH_FLOATS fp32 values (64 MiB) of device
 * memory on every GPU the library has run this call on, held until the
 * process ends.  The call itself allocates and frees nothing.
 *   Arguments, layouts, path choice and results: as clifford_block2_nd.
 *   Limit: B * C_mid * d_mid^k * N_B <= CLIFF_NOALLOC_SCRATCH_FLOATS, else
 *          CLIFF_ESCRATCH before any work is enqueued (also for blocks that
 *          would run as one fused launch and need no scratch).
 *   Sharing: every call on one GPU uses that GPU's one array (its contents are
 *          whatever the last call left; each call writes every value it
 *          reads, so nothing needs clearing).  Calls whose executions
 *          overlap on one GPU -- on different streams, or from several host
 *          threads without ordering -- race on it and give undefined results.
 *   Errors: as clifford_block2_nd, plus CLIFF_ESCRATCH, and CLIFF_EDEVICE
 *          when the array's device address cannot be obtained.
 */
#define CLIFF_NOALLOC_SCRATCH_FLOATS (16 * 1024 * 1024)
cliff_status clifford_block2_nd_noalloc(int k, const int8_t* g, int64_t B, int64_t C_in,
                                        int64_t C_mid, int64_t C_out, int64_t d_image,
                                        int64_t d_filter, const float* input,
                                        const float* filters1, const float* bias1,
                                        const cliff_act_desc* act1, const float* filters2,
                                        const float* bias2, const cliff_act_desc* act2,
                                        float* output, void* stream);

/*
 * Standalone multivector activation (paper, Algorithm 3).
 *   nb      N_B in {2, 4, 8}
 *   input   device [B, C, P, N_B]   (P positions per channel; P = 1 gives
 *           the paper's [B, C, N_B])
 *   output  device [B, C, P, N_B]; may equal input (in place) but must not
 *           overlap it otherwise
 * act must not be NULL; B, C, P >= 1 (B = 0 enqueues nothing).
 * Alignment: input and output 16-byte aligned.
 */
cliff_status multivector_act(int nb, int64_t B, int64_t C, int64_t P,
                             const cliff_act_desc* act, const float* input,
                             float* output, void* stream);

/*
 * Host-side multiplication table the kernels are driven by (paper,
 * Background, "Clifford Algebra"), for output blade i and input blade j:
 *     (w * x)_i = sum_j sign[i*N_B + j] * w_{src[i*N_B + j]} * x_j
 * i.e. e_{src} e_j = sign * e_i.  src and sign are caller-owned host arrays
 * of N_B*N_B entries; sign is in {-1, 0, +1}.  No device work.
 */
cliff_status cliffconv_cayley_table(int k, const int8_t* g, int8_t* src,
                                    int8_t* sign);

/* Static, human-readable name of a status code. */
const char* cliffconv_status_string(cliff_status s);

#ifdef __cplusplus
}
#endif

#endif /* CLIFFCONV_H */
