// tbn_quantize.hip -- per-filter discretisation (Sec. 2, Eq. 3) and optimal scale
// (Sec. 2, Eq. 4-5) as a wavefront reduction, writing the TBN2 packed codes directly.
//
// A block per filter; each of its waves walks chunks of 64 elements; lane l reads element
// 64c + l (one coalesced 256-byte row segment per chunk), takes the two
// predicates of Eq. (3) -- magnitude (|W| > 1) and sign (!(W > 0), which puts both zeros
// and -1 <= W <= 0 on the negative side) -- and the wave turns them into two 64-bit
// ballots.  Lanes 0..3 then assemble the four packed words of the chunk from the
// ballots (even elements to bytes 0/1, odd elements to bytes 2/3) and store them as one
// 16-byte segment.  The B1/B2 sums of Eq. (4)-(5) accumulate per lane in fp64, are
// reduced across each wave and then over the waves in order; |B2| is the popcount of the
// magnitude ballots.  The same kernel can first apply the SGD update to each weight (the
// update step of Algorithm 1 fused with the next iteration's quantisation).
#include "tbn_device.h"
#include "tbn_kernels.h"

namespace tbn {

// Gather the even-indexed bits of a 16-bit value into an 8-bit value.
__device__ __forceinline__ uint32_t even_bits16(uint32_t x) {
    x &= 0x5555u;
    x = (x | (x >> 1)) & 0x3333u;
    x = (x | (x >> 2)) & 0x0F0Fu;
    x = (x | (x >> 4)) & 0x00FFu;
    return x;
}

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
    return v;
}

// Momentum-SGD update of one weight (Sec. 4 optimiser), written with explicit fused
// multiply-adds so that the standalone update and the fused update-and-quantise step give
// bit-identical weights: v = momentum v + (g + decay w), w = w - lr v.
__device__ __forceinline__ void sgd_update(float& w, float& v, float g, float lr, float mu, float wd) {
    v = __builtin_fmaf(mu, v, __builtin_fmaf(wd, w, g));
    w = __builtin_fmaf(-lr, v, w);
}

// One block of four waves per filter: wave v takes the chunks c = v, v + 4, ... (four at a
// time, loads issued together), and the per-wave fp64 sums and counts are combined in wave
// order through LDS.  With SGD, each element is first updated in place (w, v from their
// gradient g) and the updated weight is what Eq. (3)-(5) see: the next iteration's
// quantisation fused into this iteration's update, one pass over the filter.
//
// Variants of the discretisation (Sec. 2 adopts the deterministic rule "for simplicity"):
//   * threshold t (QuantVariant::thr_bits, the bit pattern of t > 0): |W| > t selects the
//     magnitude 2 instead of |W| > 1;
//   * STOCH: stochastic discretisation with caller-supplied uniform numbers u in [0, 1):
//     W is clamped to [-2, 2] and rounded to one of its two neighbouring levels with the
//     probabilities that make the expected code equal W (between -1 and 1 the neighbours
//     are -1 and 1).  All decisions are fp32 comparisons.
// The scale is in every case the optimum of Eq. (4) for the chosen codes,
// alpha = sum_i W_i c_i / sum_i c_i^2, which for the deterministic rules is Eq. (5).
template <bool SGD, bool STOCH>
__global__ __launch_bounds__(256) void quantize_kernel(const float* __restrict__ w, int64_t K,
                                                       int64_t n, uint32_t* __restrict__ codes,
                                                       float* __restrict__ alpha,
                                                       int32_t* __restrict__ counts, SgdArgs sgd,
                                                       QuantVariant var) {
    __shared__ double sh1[4], sh2[4];
    __shared__ int64_t shn[4];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int64_t k = blockIdx.x;  // filter of this block
    const int64_t nb = (n + 63) / 64;
    uint32_t* out = codes + ((k / 64) * nb * 64 + (k % 64)) * 4;  // + chunk*256 per chunk
    if (k >= K) {  // padding filter of the last 64-filter block: all bits zero
        for (int64_t c = threadIdx.x; c < nb * 4; c += 256) out[(c / 4) * 256 + (c % 4)] = 0u;
        return;
    }
    const float* wk = w + k * n;
    double s1 = 0.0, s2 = 0.0;
    int64_t n2 = 0;
    for (int64_t c0 = wave; c0 < nb; c0 += 16) {
        uint32_t u[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {  // branch-free loads: out-of-range lanes read w[k][0]
            const int64_t i = (c0 + 4 * j) * 64 + lane;
            u[j] = __float_as_uint(wk[i < n ? i : 0]);
        }
        if constexpr (SGD) {
            float vv[4], gg[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int64_t i = (c0 + 4 * j) * 64 + lane;
                vv[j] = sgd.v[k * n + (i < n ? i : 0)];
                gg[j] = sgd.g[k * n + (i < n ? i : 0)];
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int64_t i = (c0 + 4 * j) * 64 + lane;
                float wf = __uint_as_float(u[j]);
                sgd_update(wf, vv[j], gg[j], sgd.lr, sgd.mu, sgd.wd);
                u[j] = __float_as_uint(wf);
                if (c0 + 4 * j < nb && i < n) {
                    sgd.w[k * n + i] = wf;
                    sgd.v[k * n + i] = vv[j];
                }
            }
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t c = c0 + 4 * j;
            if (c >= nb) break;
            const bool in = c * 64 + lane < n;
            // The predicates of Eq. (3) on the bit pattern, so that they are exact in any
            // denormal mode: |W| > 1, and W > 0 (false for both zeros and for NaN).
            const uint32_t abits = u[j] & 0x7FFFFFFFu;
            const bool nan = abits > 0x7F800000u;
            bool mag, neg;
            if constexpr (STOCH) {
                const int64_t i = c * 64 + lane;
                const float uu = var.uni[k * n + (in ? i : 0)];
                const float a = fminf(fmaxf(__uint_as_float(u[j]), -2.0f), 2.0f);
                if (nan) {
                    mag = false;
                    neg = true;
                } else if (a > 1.0f) {
                    mag = uu < a - 1.0f;
                    neg = false;
                } else if (a < -1.0f) {
                    mag = uu < -1.0f - a;
                    neg = true;
                } else {
                    mag = false;
                    neg = !(uu + uu < a + 1.0f);
                }
                mag = mag && in;
                neg = neg && in;
                if (in) {  // W_i * sign(c_i), summed per magnitude
                    const double wv = (double)__uint_as_float(u[j]);
                    const double a2 = neg ? -wv : wv;
                    if (mag) s2 += a2; else s1 += a2;
                }
            } else {
                mag = in && !nan && abits > var.thr_bits;
                neg = in && !(!nan && !(u[j] >> 31) && abits != 0u);
                if (in) {
                    const double a = (double)__uint_as_float(abits);
                    if (mag) s2 += a; else s1 += a;  // a NaN weight makes alpha NaN
                }
            }
            const uint64_t M = __ballot(mag);
            const uint64_t S = __ballot(neg);
            n2 += __popcll(M);
            if (lane < 4) {
                const uint32_t m16 = (uint32_t)(M >> (16 * lane)) & 0xFFFFu;
                const uint32_t s16 = (uint32_t)(S >> (16 * lane)) & 0xFFFFu;
                const uint32_t word = even_bits16(m16) | (even_bits16(s16) << 8) |
                                      (even_bits16(m16 >> 1) << 16) | (even_bits16(s16 >> 1) << 24);
                out[c * 256 + lane] = word;
            }
        }
    }
    s1 = wave_sum(s1);
    s2 = wave_sum(s2);
    if (lane == 0) {
        sh1[wave] = s1;
        sh2[wave] = s2;
        shn[wave] = n2;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        double t1 = 0.0, t2 = 0.0;
        int64_t tn2 = 0;
        for (int v = 0; v < 4; ++v) {
            t1 += sh1[v];
            t2 += sh2[v];
            tn2 += shn[v];
        }
        const int64_t n1 = n - tn2;
        const double a = (t1 + 2.0 * t2) / (double)(n1 + 4 * tn2);
        alpha[k] = (float)a;
        if (counts) {
            counts[2 * k] = (int32_t)n1;
            counts[2 * k + 1] = (int32_t)tn2;
        }
    }
}

hipError_t launch_quantize(const float* w, int64_t K, int64_t n, uint32_t* codes, float* alpha,
                           int32_t* counts, hipStream_t stream) {
    return launch_quantize_variant(w, K, n, QuantVariant{0x3F800000u, nullptr}, codes, alpha, counts, stream);
}

hipError_t launch_quantize_variant(const float* w, int64_t K, int64_t n, const QuantVariant& var, uint32_t* codes,
                                   float* alpha, int32_t* counts, hipStream_t stream) {
    const int64_t kpad = (K + 63) / 64 * 64;
    if (var.uni)
        hipLaunchKernelGGL((quantize_kernel<false, true>), dim3((unsigned)kpad), dim3(256), 0, stream, w, K, n, codes,
                           alpha, counts, SgdArgs{}, var);
    else
        hipLaunchKernelGGL((quantize_kernel<false, false>), dim3((unsigned)kpad), dim3(256), 0, stream, w, K, n, codes,
                           alpha, counts, SgdArgs{}, var);
    return hipGetLastError();
}

hipError_t launch_sgd_quantize(const SgdArgs& sgd, int64_t K, int64_t n, uint32_t* codes, float* alpha,
                               int32_t* counts, hipStream_t stream) {
    const int64_t kpad = (K + 63) / 64 * 64;
    hipLaunchKernelGGL((quantize_kernel<true, false>), dim3((unsigned)kpad), dim3(256), 0, stream, sgd.w, K, n,
                       codes, alpha, counts, sgd, QuantVariant{0x3F800000u, nullptr});
    return hipGetLastError();
}

}  // namespace tbn
