// Clifford linear layer (paper, Algorithm 2) as a streamed GEMM on the fp32
// matrix cores (v_mfma_f32_16x16x4_f32).
//
// With one position and one tap the layer is Y = X E^T + bias, with X the
// input as stored ([B, K], K = C_in N_B), Y the output ([B, N], N = C_out N_B)
// and E the expanded weight, E[(co, i), (ci, j)] = s(i, j) w[ci, co, i ^ j]
// (table sign and source blade as in the convolution).  B is large and N, K
// are small (the paper's linear layers have 32 channels), so:
//  * every workgroup copies the raw weight [C_in, C_out, N_B] into LDS once;
//    A fragments are read from there and the sign applied in a register, so
//    the expanded weight exists nowhere (layers of 128 or 256 columns without
//    zero signs also keep the negated weight, and each lane reads the copy
//    of its sign instead of multiplying);
//  * each wave owns whole rows of Y (a tile of 16 * NWW positions by all N
//    columns) and streams its tiles without any barrier: B fragments come from
//    HBM straight into registers, PF chunks of 16 K values ahead, across tile
//    boundaries, so one tile's loads and the previous tile's stores overlap
//    the current tile's MFMAs;
//  * the grid is persistent (as many workgroups as fit at once), each wave
//    taking every (number of waves)-th tile.
//
// K order.  A 16-byte load gives lane (n, r) = (lane % 16, lane / 16) the four
// inputs k = 16 q + 4 r .. 16 q + 4 r + 3 of its position; step t of chunk q
// multiplies component t, so MFMA K slot r of that step is k = 16 q + 4 r + t.
// The A fragment is read in the same order.
#include <stdio.h>

#include <algorithm>
#include <atomic>

#include "common.hpp"
#include "epilogue.hpp"
#include "linear_geom.hpp"

namespace cliff {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef unsigned u4 __attribute__((ext_vector_type(4)));


// NB blades; RT = N / 16 row tiles (all of them per wave); KQ = K / 16
// chunks; NWW 16-position column tiles per wave tile; PF chunks of prefetch.
// Measured on MI355X (interleaved timing, C = 32 layers): 16 accumulator
// tiles per wave at 2 waves per SIMD beat 32 tiles at 1 wave by 2-11 %; 8
// chunks of prefetch are within noise of 4; non-temporal input loads cost
// 2-30 %.
#ifndef CLIFF_LIN_CHAINS  // accumulator tiles per wave
#define CLIFF_LIN_CHAINS 16
#endif
#ifndef CLIFF_LIN_PF  // chunks of 16 K values prefetched ahead
#define CLIFF_LIN_PF 4
#endif
#ifndef CLIFF_LIN_N64_WAVES4  // N = K = 64: fewer tiles per wave at more waves per SIMD
#define CLIFF_LIN_N64_WAVES4 1
#endif
#ifndef CLIFF_LIN_N64_CHAINS  // ... that many accumulator tiles per wave (one 16-position tile)
#define CLIFF_LIN_N64_CHAINS 4
#endif
#ifndef CLIFF_LIN_N64_WAVES  // ... at that many waves per SIMD
#define CLIFF_LIN_N64_WAVES 4
#endif
#ifndef CLIFF_LIN_NEG  // negated weight copy in LDS instead of sign multiplies
#define CLIFF_LIN_NEG 1
#endif
#ifndef CLIFF_LIN_NEG8  // 8-wave workgroups for 256-column layers whose two copies need them
#define CLIFF_LIN_NEG8 1
#endif
#ifndef CLIFF_LIN_AREG  // N = K = 64: the signed A values in registers for the whole kernel
#define CLIFF_LIN_AREG 1
#endif
#ifndef CLIFF_LIN_STORE_AUX  // cache policy bits of the output stores
#define CLIFF_LIN_STORE_AUX 0
#endif
#ifndef CLIFF_LIN_WAVES  // waves per SIMD the registers are sized for
#define CLIFF_LIN_WAVES 2
#endif

// NEG: LDS holds the weight and its negation; each lane's A reads take the
// copy of its sign, so no step multiplies (signatures without zero signs).
// NT threads per workgroup (4 waves; 8 where one workgroup per CU holds
// both weight copies).
template <int NB, int RT, int KQ, int NWW, int PF, int WAVES, bool NEG, int NT = 256>
__global__ __launch_bounds__(NT, WAVES) void linear_mfma_kernel(LinArgs a)
{
    static_assert(KQ % PF == 0 && KQ >= PF, "whole prefetch rounds per tile");
    constexpr int N = 16 * RT;
    constexpr int TP = 16 * NWW;
    extern __shared__ f4 smem4[];
    float* wl = reinterpret_cast<float*>(smem4);
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int waves = blockDim.x >> 6;
    const int n = lane & 15, r = lane >> 4;
    constexpr int K = KQ * 16;

    // LDS (linear_geom.hpp): the raw weight (NEG: and its negation); then
    // the bias (zero without one), the gate coefficients and the gate biases
    // (Linear mode; zero otherwise).  The epilogue reads them from here: a
    // global load issued after the input prefetch would have to wait for all
    // of it.
    const int wfloats = lin_wfloats(a);
    float* bl = wl + lin_tail(a, NEG);
    float* cl = bl + N;
    float* gl = cl + N;
    for (int e = tid; e < a.C_in * (N / 4); e += blockDim.x) {
        const f4 v = *reinterpret_cast<const f4*>(a.w + (int64_t)e * 4);
        *reinterpret_cast<f4*>(wl + lin_w_lds(a, N, e)) = v;
        if (NEG) *reinterpret_cast<f4*>(wl + wfloats + lin_w_lds(a, N, e)) = -v;
    }
    for (int e = tid; e < N; e += blockDim.x) {
        bl[e] = a.bias ? a.bias[e] : 0.f;
        cl[e] = a.act.mode >= 0 ? gate_coef(a.act, gate_slot(a.act, e % NB), e / NB) : 0.f;
        if (e < N / NB) gl[e] = a.act.mode == CLIFF_AGG_LINEAR ? a.act.bias[e] : 0.f;
    }
    __syncthreads();

    // A fragment lane (row n of a row tile, K slot r): step t of a chunk
    // reads weight blade src(i, j) with sign s(i, j) (linear_geom.hpp; NEG:
    // from the copy of its sign)
    const int i = n % NB;
    int abase[4];
    float sg[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        sg[t] = sign_of(a.sign, i * NB + (4 * r + t) % NB);
        abase[t] = lin_a_base(a, NB, n, r, t, NEG && sg[t] < 0.f);
    }

    const int64_t stride = (int64_t)gridDim.x * waves;
    int64_t t = (int64_t)blockIdx.x * waves + wave;
    if (t >= a.n_wt) return;  // wave-uniform, after the only barrier
    // row of X for column tile nw of wave tile tt (past B: the last row,
    // loaded but never stored)
    auto xrow = [&](int64_t tt, int nw) { return a.x + lin_x_row(a, K, TP, tt, nw, n, r); };
    f4 ring[PF][NWW];
#pragma unroll
    for (int p = 0; p < PF; ++p)
#pragma unroll
        for (int nw = 0; nw < NWW; ++nw)
            ring[p][nw] = *reinterpret_cast<const f4*>(xrow(t, nw) + p * 16);
    // A values of the next step, read one step ahead
    float fa[2][RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) fa[0][rt] = wl[abase[0] + lin_a_step(a, NB, 0, rt)];
    // N = K = 64: every step's signed A values stay in registers (64 per
    // lane), read and signed once, so the tile loop has no LDS reads and no
    // multiplies
    constexpr bool AREG = CLIFF_LIN_AREG && RT * 4 * KQ <= 64;
    float areg[AREG ? 4 * KQ : 1][RT];
    if constexpr (AREG) {
#pragma unroll
        for (int s = 0; s < 4 * KQ; ++s)
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) {
                const float w = wl[abase[s % 4] + lin_a_step(a, NB, s, rt)];
                areg[s][rt] = NEG ? w : w * sg[s % 4];
            }
    }

    // One tile's K loop, fully unrolled (KQ is a compile-time constant), so
    // that the compiler's wait counts stay exact: at a loop header it would
    // have to assume the oldest state of every edge and, with the previous
    // tile's stores issued after the prefetch, wait for those stores too.
    f4 acc[RT][NWW];
    auto tile = [&](int64_t tt, int64_t tnext) {
        const float* xc[NWW];
        const float* xn[NWW];
#pragma unroll
        for (int nw = 0; nw < NWW; ++nw) {
            xc[nw] = xrow(tt, nw);
            xn[nw] = xrow(tnext, nw);
        }
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
            for (int nw = 0; nw < NWW; ++nw) acc[rt][nw] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < 4 * KQ; ++s) {
            const int q = s / 4, st = s % 4, cur = s & 1, p = q % PF;
            // this step's signed A values, then the next step's A reads
            // (step 0 of the next tile after the last) spread between this
            // step's MFMAs, so their LDS latency is hidden
            float as[RT];
            if constexpr (AREG) {
#pragma unroll
                for (int rt = 0; rt < RT; ++rt) as[rt] = areg[s][rt];
            } else {
#pragma unroll
                for (int rt = 0; rt < RT; ++rt)
                    as[rt] = NEG ? fa[cur][rt] : fa[cur][rt] * sg[st];
                const int s1 = (s + 1) % (4 * KQ);
#pragma unroll
                for (int rt = 0; rt < RT; ++rt)
                    fa[cur ^ 1][rt] = wl[abase[s1 % 4] + lin_a_step(a, NB, s1, rt)];
            }
#pragma unroll
            for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                for (int nw = 0; nw < NWW; ++nw)
                    acc[rt][nw] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                        as[rt], ring[p][nw][st], acc[rt][nw], 0, 0, 0);
            if (st == 3) {
                // refill slot p: chunk q + PF of this tile, or chunk
                // q + PF - KQ of the next one (of this one again after the
                // last tile: a harmless reload)
#pragma unroll
                for (int nw = 0; nw < NWW; ++nw) {
                    const float* src =
                        q + PF < KQ ? xc[nw] + (q + PF) * 16 : xn[nw] + (q + PF - KQ) * 16;
                    ring[p][nw] = *reinterpret_cast<const f4*>(src);
                }
            }
            if constexpr (!AREG) {
                if (!NEG) __builtin_amdgcn_sched_group_barrier(0x002, RT, 0);  // sign multiplies
#pragma unroll
                for (int rt = 0; rt < RT; ++rt) {
                    __builtin_amdgcn_sched_group_barrier(0x008, NWW, 0);  // MFMA
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);    // LDS read
                }
            }
            __builtin_amdgcn_sched_group_barrier(0x008, RT * NWW, 0);
            __builtin_amdgcn_sched_group_barrier(0x020, NWW, 0);      // global loads
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    int64_t tn = t + stride;
    tile(t, tn < a.n_wt ? tn : t);
    for (;;) {
        const bool has_next = tn < a.n_wt;
        // Epilogue: D fragment lane (n, r) holds rows 4 r .. 4 r + 3 of each
        // row tile for position column n: bias, optional activation, one
        // 16-byte store per tile (the stores drain during the next tile).
        // The bias and gate parameters are the same for every tile; an opaque
        // zero offset keeps their LDS reads here instead of in registers
        // across the tile loop.
        int opq = 0;
        __asm__ volatile("" : "+s"(opq));
        const float* ble = bl + opq;
        const float* cle = cl + opq;
        const float* gle = gl + opq;
        const bool has_act = a.act.mode >= 0;
        const bool mean = a.act.mode == CLIFF_AGG_MEAN;
        // Stores go through a buffer descriptor covering this tile's valid
        // rows: the hardware drops those past B, with no branch (a branch
        // around a store would make the compiler assume the store might not
        // have been issued and wait for the next tile's prefetch too early).
        const int64_t m0 = t * TP;
        const int64_t rows = lin_y_rows(a, TP, t);
        // (raw descriptor: stride 0, size in bytes; word 3 = 32-bit data
        // format, the value CDNA's buffer instructions expect for raw access)
        const __amdgpu_buffer_rsrc_t ydesc = __builtin_amdgcn_make_buffer_rsrc(
            a.y + m0 * N, (short)0, (int)(rows * N * 4), 0x00020000);
        // sigmoid of the gate: Linear adds the channel's bias (zero in the
        // other modes), Mean divides by the number of blades
        auto gate = [&](float sum, int co) {
            float s = sum + gle[co];
            if (mean) s = s / (float)a.act.K;
            return 1.0f / (1.0f + __expf(-s));
        };
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            const int row0 = 16 * rt + 4 * r;  // = co * NB + blade of component 0
            const f4 bb = *reinterpret_cast<const f4*>(ble + row0);
            f4 cf = f4{0.f, 0.f, 0.f, 0.f};
            if (has_act) cf = *reinterpret_cast<const f4*>(cle + row0);
#pragma unroll
            for (int nw = 0; nw < NWW; ++nw) {
                f4 v = acc[rt][nw] + bb;
                if (has_act) {
                    if constexpr (NB == 2) {
                        // two multivectors: channels row0 / 2 and row0 / 2 + 1
                        const float g0 = gate(cf[0] * v[0] + cf[1] * v[1], row0 / 2);
                        const float g1 = gate(cf[2] * v[2] + cf[3] * v[3], row0 / 2 + 1);
                        v[0] *= g0;
                        v[1] *= g0;
                        v[2] *= g1;
                        v[3] *= g1;
                    } else {
                        float part = cf[0] * v[0] + cf[1] * v[1] + cf[2] * v[2] + cf[3] * v[3];
                        // N_B = 8: the other half of the multivector is in lane ^ 16
                        if (NB == 8) part += __shfl_xor(part, 16);
                        v *= gate(part, row0 / NB);
                    }
                }
                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u4, v), ydesc,
                                                       lin_y_byte(N, nw, n, row0), 0,
                                                       CLIFF_LIN_STORE_AUX);
            }
        }
        if (!has_next) break;
        t = tn;
        tn = t + stride;
        tile(t, tn < a.n_wt ? tn : t);
    }
}

// Resident workgroups per CU of one kernel instantiation at an LDS size,
// cached per instantiation (packed (lds << 8) | occ); 0 when the query fails.
template <int NB, int RT, int KQ, int NWW, int PF, int WAVES, bool NEG, int NT = 256>
int linear_occupancy(int64_t lds)
{
    // With a launch observer (the host-side checker, no GPU): the residency
    // the launch bounds ask for (WAVES waves per SIMD), within the LDS.
    if (launch_observer)
        return lds < 1 || lds > 160 * 1024
                   ? 0
                   : (int)std::min<int64_t>(4 * WAVES * 64 / NT, 160 * 1024 / lds);
    static std::atomic<int64_t> cache{0};
    auto kern = linear_mfma_kernel<NB, RT, KQ, NWW, PF, WAVES, NEG, NT>;
    const int64_t c = cache.load(std::memory_order_relaxed);
    if ((c >> 8) == lds && (c & 0xff)) return (int)(c & 0xff);
    int occ = 0;
    if (lds > 160 * 1024 ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kern, NT, (size_t)lds) != hipSuccess ||
        occ < 1)
        return 0;
    cache.store((lds << 8) | std::min(occ, 255), std::memory_order_relaxed);
    return occ;
}

template <int NB, int RT, int KQ>
cliff_status run_linear(const ConvProblem& p, hipStream_t stream)
{
    // 16 independent accumulator tiles per wave at 2 waves per SIMD; N = K =
    // 64 (HBM-bound) does better with more waves per SIMD and fewer tiles:
    // 8 tiles at 4 waves measured +7 % on the 1-D C = 32 layer (-1 to -3 % at
    // N = 128), 4 tiles (one 16-position tile per wave) at 4 waves a further
    // +4 % (4.57 -> 4.75 TB/s at B = 2^21; the same at 6 waves per SIMD)
    constexpr bool NARROW_N = RT == 4 && KQ == 4 && CLIFF_LIN_N64_WAVES4;
    constexpr int CHAINS = NARROW_N ? CLIFF_LIN_N64_CHAINS : CLIFF_LIN_CHAINS;
    constexpr int WAVES = NARROW_N ? CLIFF_LIN_N64_WAVES : CLIFF_LIN_WAVES;
    constexpr int NWW = RT >= CHAINS ? 1 : CHAINS / RT;
    // (N = 64 with K = 256: 2 chunks, which keeps that unrolled kernel
    // within the registers of 2 waves per SIMD)
    constexpr int PF0 = CLIFF_LIN_PF < KQ ? CLIFF_LIN_PF : KQ;
    constexpr int PF = RT == 4 && KQ == 16 && PF0 > 2 ? 2 : PF0;
    constexpr int TP = 16 * NWW;
    constexpr int N = 16 * RT;
    if (p.C_out * NB != N || p.C_in * NB != 16 * KQ) return CLIFF_EUNSUPPORTED;
    // LDS pitch: the four K slots of an A read fall on different banks
    const int want = NB == 2 ? 8 : 16;
    const int WP = N + ((want - N % 64) % 64 + 64) % 64;
    const int64_t wbytes = p.C_in * (int64_t)WP * 4, tail = (2 * N + N / NB) * 4;
    const int64_t n_wt = (p.B + TP - 1) / TP;
    if (n_wt >= (1ll << 40)) return CLIFF_EUNSUPPORTED;
    auto kern = linear_mfma_kernel<NB, RT, KQ, NWW, PF, WAVES, false>;
    auto kern_neg = linear_mfma_kernel<NB, RT, KQ, NWW, PF, WAVES, true>;
    const int occ = linear_occupancy<NB, RT, KQ, NWW, PF, WAVES, false>(wbytes + tail);
    if (occ < 1) return CLIFF_EUNSUPPORTED;
    // The negated weight copy replaces the sign multiplies where no sign is
    // zero and the doubled weight keeps the same residency.  Measured
    // (interleaved): 3D C = 32 (N = 256) +3.4 %, 1-D C = 64 (N = 128)
    // +1.7 %, the other N = 128 layers within noise; the HBM-bound N = 64
    // layer -2 %, so it keeps the multiplies.
    const bool neg_ok = CLIFF_LIN_NEG && RT >= 8 && p.sign.zero == 0;
    const bool neg = neg_ok &&
                     linear_occupancy<NB, RT, KQ, NWW, PF, WAVES, true>(2 * wbytes + tail) >= occ;
    // 256-column layers whose weight copies leave room for only one 4-wave
    // workgroup per CU: 8-wave workgroups share them at twice the waves per
    // SIMD, with both copies where those fit at the 4-wave residency (64
    // input channels in 2D), else with the weight alone where it holds a CU
    // to one 4-wave workgroup (128 input channels in 1-D)
    int occ8 = 0;
    bool neg8 = false, plain8 = false;
    if constexpr (RT == 16 && KQ == 16 && CLIFF_LIN_NEG8) {
        if (neg_ok && !neg) {
            occ8 = linear_occupancy<NB, RT, KQ, NWW, PF, WAVES, true, 512>(2 * wbytes + tail);
            neg8 = occ8 > 0 && 2 * occ8 >= occ;
        }
        if (!neg && !neg8 && occ == 1) {
            occ8 = linear_occupancy<NB, RT, KQ, NWW, PF, WAVES, false, 512>(wbytes + tail);
            plain8 = occ8 >= 1;
        }
    }
    const int64_t lds = (neg || neg8 ? 2 : 1) * wbytes + tail;
    const int cus = device_cus();
    if (cus < 1) return CLIFF_EDEVICE;
    const int wg_waves = neg8 || plain8 ? 8 : 4;
    const int64_t n_wg = std::min<int64_t>((n_wt + wg_waves - 1) / wg_waves,
                                           (int64_t)cus * (neg8 || plain8 ? occ8 : occ));

    LinArgs a;
    a.x = p.x;
    a.w = p.w;
    a.bias = p.bias;
    a.y = p.y;
    a.B = p.B;
    a.n_wt = n_wt;
    a.C_in = (int)p.C_in;
    a.WP = WP;
    a.sign = p.sign;
    a.act = p.act;
    if (debug_enabled())
        fprintf(stderr,
                "cliffconv: linear_mfma N_B=%d N=%d K=%d, %d positions per wave tile, "
                "%lld wave tiles, %lld workgroups of %d waves (%d per CU), %lld LDS bytes%s\n",
                NB, N, 16 * KQ, TP, (long long)n_wt, (long long)n_wg, wg_waves,
                neg8 || plain8 ? occ8 : occ, (long long)lds,
                neg || neg8 ? ", negated weight copy" : "");
    if constexpr (RT == 16 && KQ == 16 && CLIFF_LIN_NEG8) {
        if (neg8 || plain8) {
            if (observe_launch(LAUNCH_LINEAR_MFMA, {NB, RT, KQ, NWW, PF, WAVES, neg8, 512}, n_wg,
                               512, lds, &a))
                return CLIFF_OK;
            clear_hip_error();
            if (neg8)
                hipLaunchKernelGGL((linear_mfma_kernel<NB, RT, KQ, NWW, PF, WAVES, true, 512>),
                                   dim3((unsigned)n_wg), dim3(512), (size_t)lds, stream, a);
            else
                hipLaunchKernelGGL((linear_mfma_kernel<NB, RT, KQ, NWW, PF, WAVES, false, 512>),
                                   dim3((unsigned)n_wg), dim3(512), (size_t)lds, stream, a);
            return hipGetLastError() == hipSuccess ? CLIFF_OK : CLIFF_EDEVICE;
        }
    }
    if (observe_launch(LAUNCH_LINEAR_MFMA, {NB, RT, KQ, NWW, PF, WAVES, neg, 256}, n_wg, 256, lds,
                       &a))
        return CLIFF_OK;
    clear_hip_error();
    hipLaunchKernelGGL(neg ? kern_neg : kern, dim3((unsigned)n_wg), dim3(256), (size_t)lds,
                       stream, a);
    return hipGetLastError() == hipSuccess ? CLIFF_OK : CLIFF_EDEVICE;
}

template <int NB, int RT>
cliff_status run_linear_k(const ConvProblem& p, hipStream_t stream, int64_t kq)
{
    if (kq == 4) return run_linear<NB, RT, 4>(p, stream);
    if (kq == 8) return run_linear<NB, RT, 8>(p, stream);
    if (kq == 16) return run_linear<NB, RT, 16>(p, stream);
    return CLIFF_EUNSUPPORTED;
}

template <int NB>
cliff_status run_linear_nk(const ConvProblem& p, hipStream_t stream)
{
    const int64_t rt = p.C_out * NB / 16, kq = p.C_in * NB / 16;
    if (p.C_out * NB % 16 != 0 || p.C_in * NB % 16 != 0) return CLIFF_EUNSUPPORTED;
    if (rt == 4) return run_linear_k<NB, 4>(p, stream, kq);
    if (rt == 8) return run_linear_k<NB, 8>(p, stream, kq);
    if (rt == 16) return run_linear_k<NB, 16>(p, stream, kq);
    return CLIFF_EUNSUPPORTED;
}

}  // namespace

// Layers whose C_out N_B and C_in N_B are each 64, 128 or 256, i.e. 32, 64
// or 128 channels (k = 1), 16, 32 or 64 (k = 2), 8, 16 or 32 (k = 3).
cliff_status launch_linear_mfma(const ConvProblem& p, hipStream_t stream)
{
    if (p.d_image != 1 || p.d_filter != 1) return CLIFF_EUNSUPPORTED;
    switch (p.nb) {
        case 2: return run_linear_nk<2>(p, stream);
        case 4: return run_linear_nk<4>(p, stream);
        case 8: return run_linear_nk<8>(p, stream);
    }
    return CLIFF_EUNSUPPORTED;
}

}  // namespace cliff
