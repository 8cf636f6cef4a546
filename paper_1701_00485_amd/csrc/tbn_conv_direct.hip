// tbn_conv_direct.hip -- forward pass of a small two-bit layer (Sec. 2 Eq. 1) whose filters
// span few input channels (3x3, 5x5, 7x7 or 1x1 shapes compiled, at most 147 elements):
// single-channel MNIST-shaped layers, the first 3x3 layer over RGB and the 7x7 RGB stem at
// batch 1.  Such a layer is a few hundred MFLOP at most, so the matrix cores
// buy nothing; what costs time is latency (filter decode, input gather, output store in
// sequence).  Here every thread owns one output pixel and 8 consecutive filters:
//   * a block (four waves) covers 64 pixels and 32 filters; its filters are decoded once
//     from the packed codes into LDS as bf16 +-1 / +-2, two consecutive elements per 32-bit
//     word (pair-major, so the 8 weight pairs a thread needs for two elements are one
//     32-byte broadcast read: every lane of a wave reads the same filters);
//   * the four waves need the same 64 pixels' inputs, so each loads only every fourth
//     filter row of the patches (zero outside the image; fp32 input rounded to bf16, nearest
//     even, as in every other forward kernel) and writes it to LDS as bf16 pairs: a quarter
//     of the load instructions of per-wave gathers, which bounded the kernel (ResNet stem at
//     batch 1: 16.8 -> 11.9 us);
//   * the thread issues its loads of the filter codes, then those of its patch rows; the
//     block decodes its filters as soon as the codes land and stores the patches, and after
//     one barrier every thread accumulates its pixel two elements at a time with
//     v_dot2_f32_bf16 (an input pair read from LDS against a pair of weights: products exact,
//     sums fp32); against one fp32 FMA per element this halves both the vector instructions
//     and the LDS broadcast bytes;
//   * alpha (the column scale) and the optional scale, bias, residual and ReLU are applied
//     in fp32 and the 8 outputs written with 16-byte stores.
#include "tbn_device.h"
#include "tbn_kernels.h"

namespace tbn {

namespace {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// the word as a bf16 pair (taken by value: a bit cast applied to a vector element in place
// reads the vector's first element)
__device__ __forceinline__ bf16x2 as_bf16x2(uint32_t v) { return __builtin_bit_cast(bf16x2, v); }

constexpr int DPIX = 64;   // output pixels per block (one per lane)
constexpr int DFB = 32;    // filters per block (8 per wave)
constexpr int DMAXN = 147;  // filter elements R*S*C

// R x S filters over C channels (compile-time, so that the gather below is fully unrolled and
// all of a thread's input loads are in flight together)
template <int R, int S, int C, bool X32>
__global__ __launch_bounds__(256) void conv_direct_kernel(const ConvGemmArgs a) {
    constexpr int n = R * S * C;
    constexpr int np = (n + 1) / 2;  // element pairs (the last one zero-padded for odd n)
    static_assert(n <= DMAXN, "filter elements");
    constexpr int PW2 = np % 2 == 1 ? np : np + 1;  // words per pixel row of xs
    __shared__ __attribute__((aligned(16))) uint32_t wl[np * DFB];  // [pair][filter], bf16 x 2
    __shared__ uint32_t xs[DPIX * PW2];                               // [pixel][pair], bf16 x 2
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int grp = __builtin_amdgcn_readfirstlane(tid >> 6);  // filter group of the wave
    constexpr int nchunks = (n + 63) / 64;
    const int kb0 = blockIdx.y * DFB;

    // the block's filters: element e of filter kb0 + f is bit (e % 16) / 2 (+ 16 for odd e)
    // of word (e % 64) / 16 of the filter's 16-byte code row in chunk e / 64 (magnitude),
    // the bit 8 above it the sign, so both elements of pair j (2 j and 2 j + 1) sit in one
    // word; weights of filters past Kf are zero.  The code loads go out first, so that the
    // decode waits for them alone (vector loads complete in order).
    constexpr int DITER = (np * DFB + 255) / 256;
    uint32_t cw[DITER];
#pragma unroll
    for (int it = 0; it < DITER; ++it) {
        const int i = tid + 256 * it;
        const int e = 2 * (i >> 5), k = kb0 + (i & (DFB - 1));
        cw[it] = i < np * DFB && k < a.Kf
                     ? a.codes[((int64_t)((k >> 6) * nchunks + (e >> 6)) * 64 + (k & 63)) * 4 + ((e & 63) >> 4)]
                     : 0u;
    }

    // the pixel of lane l of every wave is pixel l of the block (zero outside the image)
    const int64_t M = (int64_t)a.N * a.P * a.Q;
    const int64_t m = (int64_t)blockIdx.x * DPIX + lane;
    const bool live = m < M;
    const uint32_t mm = live ? (uint32_t)m : 0u;  // < 2^31, checked by the host
    const uint32_t img = fdiv(mm, a.div_pq);
    const uint32_t pq = mm - img * (uint32_t)(a.P * a.Q);
    const uint32_t p = fdiv(pq, a.div_q);
    const uint32_t q = pq - p * (uint32_t)a.Q;
    const int h0 = (int)p * a.sh - a.ph, w0 = (int)q * a.sw - a.pw;
    // element index of tap (0, 0) (x has fewer than 2^31 elements, checked by the host; it
    // may be negative here, only in-image taps are used)
    const int32_t pix0 = (((int32_t)img * a.H + h0) * a.W + w0) * C;
    // unconditional gather through a buffer resource: an out-of-image tap gets an offset
    // beyond the buffer and the hardware returns zero, so no load sits behind a branch
    constexpr int ESZ = X32 ? 4 : 2;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<void*>(a.x), (short)0, (int)((int64_t)a.N * a.H * a.W * C * ESZ), 0x00020000);
    // the block's 64 pixels' inputs are loaded once, patch row r by wave r % 4 (raw bf16, fp32
    // input rounded to bf16 at once, nearest even, as in every other forward kernel), and
    // written to LDS as bf16 pairs, one row of PW2 words per pixel (PW2 odd: the 64 lanes'
    // reads of one pair fall in distinct banks)
    constexpr int RW = (R + 3) / 4;  // patch rows per wave at most
    uint32_t xv[RW * S * C];
#pragma unroll
    for (int i = 0; i < RW; ++i) {
        const int r = grp + 4 * i;
        if (r < R) {
#pragma unroll
            for (int s_ = 0; s_ < S; ++s_) {
                const bool ok = live && (unsigned)(h0 + r) < (unsigned)a.H && (unsigned)(w0 + s_) < (unsigned)a.W;
                const int off = ok ? (pix0 + (r * a.W + s_) * C) * ESZ : (int)0x80000000;
#pragma unroll
                for (int c = 0; c < C; ++c) {
                    if constexpr (X32)
                        xv[(i * S + s_) * C + c] = __builtin_amdgcn_raw_buffer_load_b32(rs, off, c * 4, 0);
                    else
                        xv[(i * S + s_) * C + c] = __builtin_amdgcn_raw_buffer_load_b16(rs, off, c * 2, 0);
                }
            }
        }
    }
#pragma unroll
    for (int it = 0; it < DITER; ++it) {
        const int i = tid + 256 * it;
        if (i < np * DFB) {
            const int e = 2 * (i >> 5);
            const int jj = (e & 15) >> 1;
            // bf16 of +-1 / +-2: 0x3F80 or 0x4000 for the magnitude bit, 0x8000 for the sign;
            // a filter past Kf has an all-zero code word but must weigh zero, as must the
            // padding element of an odd n
            auto wbits = [&](int hh) -> uint32_t {
                const uint32_t mag = (cw[it] >> (16 * hh + jj)) & 1u, sg = (cw[it] >> (16 * hh + 8 + jj)) & 1u;
                return (mag ? 0x4000u : 0x3F80u) | (sg << 15);
            };
            const bool live_k = kb0 + (i & (DFB - 1)) < a.Kf;
            const uint32_t lo = live_k ? wbits(0) : 0u;
            const uint32_t hi = live_k && e + 1 < n ? wbits(1) : 0u;
            wl[i] = lo | (hi << 16);
        }
    }
    uint16_t* xrow16 = reinterpret_cast<uint16_t*>(xs + lane * PW2);
#pragma unroll
    for (int i = 0; i < RW; ++i) {
        const int r = grp + 4 * i;
        if (r < R) {
#pragma unroll
            for (int j = 0; j < S * C; ++j) {
                const uint32_t v = xv[i * S * C + j];
                xrow16[r * S * C + j] = (uint16_t)(X32 ? f32_to_bf16_bits(__uint_as_float(v)) : v);
            }
        }
    }
    if (n % 2 == 1 && grp == 0) xrow16[n] = 0;  // the padding element of the last pair
    __syncthreads();

    const int k0 = kb0 + 8 * grp;
    if (!live || k0 >= a.Kf) return;  // no barrier follows

    float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    const uint32_t* wg = wl + 8 * grp;
    const uint32_t* xrow = xs + lane * PW2;
#pragma unroll
    for (int j2 = 0; j2 < np; ++j2) {
        // weights read two pairs at a time (the fence keeps the compiler from hoisting all
        // of them, which would cost ~150 registers and occupancy)
        if (j2 % 2 == 0) __builtin_amdgcn_sched_barrier(0);
        // the 8 weight pairs of elements 2 j2, 2 j2 + 1: the same address in every lane
        const u32x4 lo = *reinterpret_cast<const u32x4*>(wg + j2 * DFB);
        const u32x4 hi = *reinterpret_cast<const u32x4*>(wg + j2 * DFB + 4);
        const bf16x2 xp = as_bf16x2(xrow[j2]);
        acc[0] = __builtin_amdgcn_fdot2_f32_bf16(xp, as_bf16x2(lo.x), acc[0], false);
        acc[1] = __builtin_amdgcn_fdot2_f32_bf16(xp, as_bf16x2(lo.y), acc[1], false);
        acc[2] = __builtin_amdgcn_fdot2_f32_bf16(xp, as_bf16x2(lo.z), acc[2], false);
        acc[3] = __builtin_amdgcn_fdot2_f32_bf16(xp, as_bf16x2(lo.w), acc[3], false);
        acc[4] = __builtin_amdgcn_fdot2_f32_bf16(xp, as_bf16x2(hi.x), acc[4], false);
        acc[5] = __builtin_amdgcn_fdot2_f32_bf16(xp, as_bf16x2(hi.y), acc[5], false);
        acc[6] = __builtin_amdgcn_fdot2_f32_bf16(xp, as_bf16x2(hi.z), acc[6], false);
        acc[7] = __builtin_amdgcn_fdot2_f32_bf16(xp, as_bf16x2(hi.w), acc[7], false);
        if (j2 % 2 == 1 || j2 == np - 1) {
            // the sums so far are materialised here, so the products cannot be moved past
            // the next reads (which would keep every weight of the filter live at once)
#pragma unroll
            for (int j = 0; j < 8; ++j) asm volatile("" : "+v"(acc[j]));
        }
    }

    // ---- epilogue: y = act(acc * alpha * scale + bias + residual) ----
    const int Kf = a.Kf;
    const int64_t o = m * Kf + k0;
    float v8[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const int col = k0 + j < Kf ? k0 + j : Kf - 1;  // past Kf: computed, never stored
        float sc = a.colscale ? a.colscale[col] : 1.0f;
        if (a.scale) sc *= a.scale[col];
        v8[j] = acc[j] * sc + (a.bias ? a.bias[col] : 0.0f);
    }
    const bool full = k0 + 8 <= Kf && Kf % 8 == 0;  // 16-byte aligned group of 8 real columns
    if (a.residual) {
#pragma unroll
        for (int j = 0; j < 8; ++j)
            if (k0 + j < Kf)
                v8[j] += a.y_f32 ? reinterpret_cast<const float*>(a.residual)[o + j]
                                 : bf16_bits_to_f32(reinterpret_cast<const uint16_t*>(a.residual)[o + j]);
    }
    if (a.relu) {
#pragma unroll
        for (int j = 0; j < 8; ++j) v8[j] = fmaxf(v8[j], 0.0f);
    }
    if (a.y_f32) {
        float* yp = reinterpret_cast<float*>(a.y) + o;
        if (full) {
            *reinterpret_cast<f32x4*>(yp) = f32x4{v8[0], v8[1], v8[2], v8[3]};
            *reinterpret_cast<f32x4*>(yp + 4) = f32x4{v8[4], v8[5], v8[6], v8[7]};
        } else {
            for (int j = 0; j < 8 && k0 + j < Kf; ++j) yp[j] = v8[j];
        }
    } else {
        uint16_t* yp = reinterpret_cast<uint16_t*>(a.y) + o;
        if (full) {
            *reinterpret_cast<u32x4*>(yp) = u32x4{pack_bf16x2(v8[0], v8[1]), pack_bf16x2(v8[2], v8[3]),
                                                  pack_bf16x2(v8[4], v8[5]), pack_bf16x2(v8[6], v8[7])};
        } else {
            for (int j = 0; j < 8 && k0 + j < Kf; ++j) yp[j] = (uint16_t)f32_to_bf16_bits(v8[j]);
        }
    }
}

}  // namespace

// filter shapes with a compiled kernel: 3x3 over 1..7 channels, 5x5 over 1..2, 7x7 over 1 and
// 3, 1x1 over 1..8
static const void* direct_kernel(int R, int S, int C, bool x32) {
#define TBN_D(r, s, c) \
    if (R == r && S == s && C == c) \
        return x32 ? reinterpret_cast<const void*>(&conv_direct_kernel<r, s, c, true>) \
                   : reinterpret_cast<const void*>(&conv_direct_kernel<r, s, c, false>);
    TBN_D(3, 3, 1) TBN_D(3, 3, 2) TBN_D(3, 3, 3) TBN_D(3, 3, 4) TBN_D(3, 3, 5) TBN_D(3, 3, 6) TBN_D(3, 3, 7)
    TBN_D(5, 5, 1) TBN_D(5, 5, 2) TBN_D(7, 7, 1) TBN_D(7, 7, 3)
    TBN_D(1, 1, 1) TBN_D(1, 1, 2) TBN_D(1, 1, 3) TBN_D(1, 1, 4) TBN_D(1, 1, 5) TBN_D(1, 1, 6) TBN_D(1, 1, 7)
    TBN_D(1, 1, 8)
#undef TBN_D
    return nullptr;
}

bool conv_direct_eligible(const ConvGemmArgs& a) {
    // forward pass with packed codes, a compiled filter shape (at most 147 elements, C <= 8),
    // and little work in total (at most 2^28 multiply-adds: beyond that the matrix-core
    // kernels win; the 7x7 RGB stem, 1.2e8 multiply-adds per image, measured 12 against 22 us
    // on the thin kernel at batch 1, 17 against 22 at batch 2)
    const int64_t n = (int64_t)a.R * a.S * a.C;
    const int64_t macs = (int64_t)a.N * a.P * a.Q * a.Kf * n;
    return !a.apair && !a.wdense && direct_kernel(a.R, a.S, a.C, a.x_f32 != 0) != nullptr &&
           macs <= (1ll << 28) && (int64_t)a.N * a.P * a.Q < 0x7FFFFFFFll &&
           (int64_t)a.N * a.H * a.W * a.C < 0x7FFFFFFFll;
}

hipError_t launch_conv_direct(const ConvGemmArgs& a, hipStream_t stream) {
    const void* fn = direct_kernel(a.R, a.S, a.C, a.x_f32 != 0);
    if (!fn) return hipErrorInvalidValue;
    const int64_t M = (int64_t)a.N * a.P * a.Q;
    const dim3 grid((unsigned)((M + DPIX - 1) / DPIX), (unsigned)((a.Kf + DFB - 1) / DFB));
    ConvGemmArgs ka = a;
    void* args[] = {&ka};
    return hipLaunchKernel(fn, grid, dim3(256), args, 0, stream);
}

}  // namespace tbn
