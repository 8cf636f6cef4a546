// tbn_fc_stream.hip -- forward pass of a two-bit fully-connected layer (Sec. 2 Eq. 1 with
// the whole input as one filter window) for a small batch (N <= 16): the weight-streaming
// regime, where the packed codes (0.25 byte per weight) are the only large operand and HBM
// bandwidth, not arithmetic, sets the speed.
//
//   * a block of 4 waves owns the 64 filters of one 1 KiB-per-64-elements code block row;
//     wave w takes filters 16 w .. 16 w + 15 as the 16 rows of v_mfma_f32_16x16x32_bf16,
//     the batch is its 16 columns (columns >= N unused);
//   * lane (f = lane % 16, g = lane / 16) loads, per step, the four code words of filter f
//     in element block ib + g (16 bytes; the 64 lanes read four 256-byte runs);
//   * the reduction order is permuted so that each lane feeds the MFMA only from its own
//     words: MFMA s (s = 0..7) of a step takes, from lane group g, elements 8 s .. 8 s + 7
//     of block ib + g, and the activation operand reads the same elements from LDS;
//   * codes are decoded in registers to exact bf16 +-0.5/+-1 (half the code: the pair
//     comes from one shift and one and-or, against three ops for +-1/+-2), and 2 alpha
//     scales the fp32 sum (exact); the loads of the next steps are issued before the
//     MFMAs of the current ones (several buffers of loads in flight per wave), and four
//     accumulators keep four MFMA chains in flight;
//   * the activations of the batch (N x n bf16) sit in LDS, zero-padded to whole steps,
//     plus one zero row that the unused batch columns read (no branch per read; those
//     output columns are never stored);
//   * alpha, the optional scale / bias / residual / ReLU are applied to the fp32 sums.
#include "tbn_device.h"
#include "tbn_kernels.h"

namespace tbn {

namespace {

typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4_t mfma16(bf16x8 a, bf16x8 b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// (t << SH) | base in one v_lshl_or_b32 (the compiler splits it into two VOP2 ops to keep
// its literal operands; with base in an SGPR the VOP3 form needs none).
template <int SH>
__device__ __forceinline__ uint32_t lshl_or(uint32_t t, uint32_t base) {
    uint32_t r;
    asm("v_lshl_or_b32 %0, %1, %2, %3" : "=v"(r) : "v"(t), "n"(SH), "s"(base));
    return r;
}

// Elements 8 h .. 8 h + 7 of a packed word as bf16 code / 2: pair j moves the magnitude
// bits (bit j of bytes 0 and 2) to bit 7 of each half and the sign bits (bytes 1 and 3)
// to bit 15, over 0.5 = 0x3F00 (bit 7 clear, so the magnitude bit makes 1.0 by an or):
// one and and one shift-or per pair.
template <int H>
__device__ __forceinline__ bf16x8 decode8_half(uint32_t w, uint32_t base) {
    u32x4 r;
    r[0] = lshl_or<7 - 4 * H>(w & (0x01010101u << (4 * H)), base);
    r[1] = lshl_or<6 - 4 * H>(w & (0x01010101u << (4 * H + 1)), base);
    r[2] = lshl_or<5 - 4 * H>(w & (0x01010101u << (4 * H + 2)), base);
    r[3] = lshl_or<4 - 4 * H>(w & (0x01010101u << (4 * H + 3)), base);
    return as_bf16x8(r);
}

// KU code loads (16 bytes per lane) per buffer, NBUF buffers in flight per wave; G groups
// of four waves per block, group g reducing the g-th of G equal ranges of steps (more waves
// per SIMD to keep loads in flight, no partial sums in memory: the groups add through LDS).
template <int KU, int NBUF, int G>
__global__ __launch_bounds__(256 * G) void fc_stream_kernel(const ConvGemmArgs a, int32_t n, int32_t nsteps,
                                                            int32_t xpitch) {
    extern __shared__ __attribute__((aligned(16))) uint16_t xl[];  // [N + 1][xpitch] bf16, then group sums
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = (tid >> 6) & 3;
    const int grp = G > 1 ? __builtin_amdgcn_readfirstlane(tid >> 8) : 0;
    const int steps_g = nsteps / G;       // steps of each group (the host pads to a multiple)
    const int step_base = grp * steps_g;
    const int N = a.N;
    const int K = a.Kf;
    const int NB = (n + 63) / 64;  // element blocks of a filter row


    const int f = lane & 15, g = lane >> 4;
    const int kb = blockIdx.x;              // 64-filter block
    const int fr = 16 * wave + f;           // filter row inside the block
    const u32x4* codes = reinterpret_cast<const u32x4*>(a.codes) + ((int64_t)kb * NB * 64 + fr);
    // activation operand: batch column f of lane group g (the zero row for columns >= N)
    const uint16_t* xrow = xl + (f < N ? f : N) * xpitch;

    // four accumulators in rotation keep four independent MFMA chains in flight
    f32x4_t acc[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[i] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
    u32x4 wbuf[NBUF][KU];
    auto load = [&](u32x4 (&w)[KU], int step0) {
#pragma unroll
        for (int u = 0; u < KU; ++u) {
            int ib = 4 * (step_base + step0 + u) + g;
            ib = ib < NB ? ib : NB - 1;  // in bounds; its activations are zero past n
            w[u] = __builtin_nontemporal_load(&codes[(int64_t)ib * 64]);  // read once: streaming
        }
    };
    const uint32_t half_one = __builtin_amdgcn_readfirstlane(0x3F003F00u);  // bf16 (0.5, 0.5)
    auto compute = [&](const u32x4 (&w)[KU], int step0) {
#pragma unroll
        for (int u = 0; u < KU; ++u) {
            const uint16_t* xb = xrow + (4 * (step_base + step0 + u) + g) * 64;
            bf16x8 bx[8];  // the step's activation operands, read before its MFMAs
#pragma unroll
            for (int s = 0; s < 8; ++s) bx[s] = *reinterpret_cast<const bf16x8*>(xb + 8 * s);
#pragma unroll
            for (int s = 0; s < 8; s += 2) {
                acc[s & 3] = mfma16(decode8_half<0>(w[u][s >> 1], half_one), bx[s], acc[s & 3]);
                acc[(s + 1) & 3] = mfma16(decode8_half<1>(w[u][s >> 1], half_one), bx[s + 1], acc[(s + 1) & 3]);
            }
        }
    };
    // ---- the batch's activations into LDS (zero beyond n, and the zero row).  When they
    //      fit one pass of 16-byte pieces (8 per thread), their loads are issued before the
    //      first code loads, so that writing them to LDS waits only for them (loads complete
    //      in order) and the code loads stay in flight across the barrier ----
    const int pieces = (N + 1) * xpitch / 8;
    const int ppr = xpitch / 8;  // pieces per row
    const bool x_one_pass = !a.x_f32 && n % 8 == 0 && pieces <= 256 * G * 8;
    u32x4 xv[8];
    if (x_one_pass) {
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int i = tid + 256 * G * u;
            const int r = i / ppr, e = (i - r * ppr) * 8;
            const bool ok = i < pieces && r < N && e < n;
            xv[u] = ok ? *reinterpret_cast<const u32x4*>(reinterpret_cast<const uint16_t*>(a.x) + (int64_t)r * n + e)
                       : u32x4{0u, 0u, 0u, 0u};
        }
    }
    // nsteps is a multiple of NBUF KU (the host pads the activations in LDS to match); the
    // first code loads are in flight while the activations are staged
#pragma unroll
    for (int b = 0; b < NBUF; ++b) load(wbuf[b], b * KU);
    if (x_one_pass) {
#pragma unroll
        for (int u = 0; u < 8; ++u)
            if (tid + 256 * G * u < pieces) reinterpret_cast<u32x4*>(xl)[tid + 256 * G * u] = xv[u];
    } else if (!a.x_f32 && n % 8 == 0) {
        // 16-byte pieces, the loads of a thread issued together
        for (int i0 = tid; i0 < pieces; i0 += 256 * G * 8) {
            u32x4 v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int i = i0 + 256 * G * u;
                const int r = i / ppr, e = (i - r * ppr) * 8;
                const bool ok = i < pieces && r < N && e < n;
                v[u] = ok ? *reinterpret_cast<const u32x4*>(reinterpret_cast<const uint16_t*>(a.x) + (int64_t)r * n + e)
                          : u32x4{0u, 0u, 0u, 0u};
            }
#pragma unroll
            for (int u = 0; u < 8; ++u)
                if (i0 + 256 * G * u < pieces) reinterpret_cast<u32x4*>(xl)[i0 + 256 * G * u] = v[u];
        }
    } else {
        for (int i = tid; i < (N + 1) * xpitch; i += 256 * G) {
            const int r = i / xpitch, e = i - (i / xpitch) * xpitch;
            uint16_t v = 0;
            if (e < n && r < N)
                v = a.x_f32 ? (uint16_t)f32_to_bf16_bits(reinterpret_cast<const float*>(a.x)[(int64_t)r * n + e])
                            : reinterpret_cast<const uint16_t*>(a.x)[(int64_t)r * n + e];
            xl[i] = v;
        }
    }
    __syncthreads();
    for (int st = 0; st < steps_g; st += NBUF * KU) {
#pragma unroll
        for (int b = 0; b < NBUF; ++b) {
            compute(wbuf[b], st + b * KU);
            if (st + (NBUF + b) * KU < steps_g) load(wbuf[b], st + (NBUF + b) * KU);
        }
    }
    f32x4_t t = (acc[0] + acc[1]) + (acc[2] + acc[3]);
    if constexpr (G > 1) {
        // groups 1 .. G-1 hand their sums to group 0, which adds them in group order
        f32x4_t* xs = reinterpret_cast<f32x4_t*>(xl + (N + 1) * xpitch);
        if (grp > 0) xs[((grp - 1) * 4 + wave) * 64 + lane] = t;
        __syncthreads();
        if (grp > 0) return;  // no barrier follows
#pragma unroll
        for (int gg = 1; gg < G; ++gg) t += xs[((gg - 1) * 4 + wave) * 64 + lane];
    }

    // ---- epilogue: lane holds batch column f, filters 4 g .. 4 g + 3 of the wave's 16 ----
    if (f >= N) return;
    const int k0 = kb * 64 + 16 * wave + 4 * g;
    float v4[4] = {t.x, t.y, t.z, t.w};
    const int64_t o = (int64_t)f * K + k0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int k = k0 + e;
        if (k >= K) break;
        float sc = 2.0f * (a.colscale ? a.colscale[k] : 1.0f);  // the codes were decoded halved
        if (a.scale) sc *= a.scale[k];
        float v = v4[e] * sc + (a.bias ? a.bias[k] : 0.0f);
        if (a.residual)
            v += a.y_f32 ? reinterpret_cast<const float*>(a.residual)[o + e]
                         : bf16_bits_to_f32(reinterpret_cast<const uint16_t*>(a.residual)[o + e]);
        if (a.relu) v = fmaxf(v, 0.0f);
        if (a.y_f32)
            reinterpret_cast<float*>(a.y)[o + e] = v;
        else
            reinterpret_cast<uint16_t*>(a.y)[o + e] = (uint16_t)f32_to_bf16_bits(v);
    }
}

}  // namespace

// (loads per buffer, buffers, groups) of each variant; the tuning knob selects one for
// sweeps.  Measured on the 8192 -> 32768 batch-1 layer, graph-replayed, alternating in one
// process, with the activations staged ahead of the first code loads: one group with four
// buffers of two 16-byte loads 17.5-17.7 us per call (the default, variant 0), two groups
// with two buffers of four 17.8-18.4 us, two groups with four buffers of two 18.0-18.7 us,
// four groups ~20 us (one block per CU).
constexpr int kNumVariants = 8;
constexpr int kVariants[kNumVariants][3] = {{2, 4, 1}, {4, 2, 1}, {8, 2, 1}, {4, 3, 1},
                                            {2, 4, 2}, {4, 2, 2}, {2, 2, 4}, {2, 3, 2}};

bool fc_stream_plan(const ConvGemmArgs& a, FcStreamPlan* p) {
    // a fully-connected layer: the filter window covers the whole (unpadded) input map
    if (a.apair || a.N > 16 || a.P != 1 || a.Q != 1 || a.R != a.H || a.S != a.W || a.ph != 0 || a.pw != 0)
        return false;
    const int forced = knob(KNOB_FC_VARIANT);
    p->variant = forced >= 0 && forced < kNumVariants ? forced : 0;
    const int64_t n = (int64_t)a.R * a.S * a.C;
    const int64_t nb = (n + 63) / 64;
    const int G = kVariants[p->variant][2];
    // element blocks per iteration of every group
    const int64_t per = 4 * kVariants[p->variant][0] * kVariants[p->variant][1] * G;
    const int64_t steps_blocks = (nb + per - 1) / per * per;
    const int64_t xpitch = steps_blocks * 64;
    // + the zero row, then the group sums (16 bytes per lane of groups 1 .. G-1)
    const int64_t lds = (int64_t)(a.N + 1) * xpitch * 2 + (int64_t)(G - 1) * 256 * 16;
    if (lds > 64 * 1024 || n > (1 << 24)) return false;
    p->n = (int32_t)n;
    p->nsteps = (int32_t)(steps_blocks / 4);
    p->xpitch = (int32_t)xpitch;
    p->lds_bytes = (int32_t)lds;
    return true;
}

hipError_t launch_fc_stream(const ConvGemmArgs& a, const FcStreamPlan& p, hipStream_t stream) {
    const dim3 grid((unsigned)((a.Kf + 63) / 64));
#define TBN_FC(ku, nb, g) \
    hipLaunchKernelGGL((fc_stream_kernel<ku, nb, g>), grid, dim3(256 * g), p.lds_bytes, stream, a, p.n, p.nsteps, p.xpitch)
    switch (p.variant) {
        case 1: TBN_FC(4, 2, 1); break;
        case 2: TBN_FC(8, 2, 1); break;
        case 3: TBN_FC(4, 3, 1); break;
        case 4: TBN_FC(2, 4, 2); break;
        case 6: TBN_FC(2, 2, 4); break;
        case 7: TBN_FC(2, 3, 2); break;
        case 0: TBN_FC(2, 4, 1); break;
        default: TBN_FC(4, 2, 2); break;
    }
#undef TBN_FC
    return hipGetLastError();
}

}  // namespace tbn
