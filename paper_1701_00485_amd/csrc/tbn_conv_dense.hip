// tbn_conv_dense.hip -- forward convolution with real-valued filters (Eq. 1 without the
// two-bit approximation), for a layer kept in full precision such as the first convolution
// of a CIFAR-shaped network, whose three input channels make it a small share of the work.
//
// Filters arrive as fp32 [K][R][S][C] and are rounded to bf16 (nearest even) as they are
// staged in LDS, activations are bf16 (or fp32 rounded the same way); products accumulate
// in fp32.  One thread computes 16 filters of one output pixel; the block's 16 filters of
// up to 512 reduction elements sit in LDS, read as broadcasts.
#include "tbn_device.h"
#include "tbn_kernels.h"

namespace tbn {

namespace {

constexpr int kDenseFilters = 16;
constexpr int kDenseChunk = 512;  // reduction elements per LDS fill (32 KiB)

__device__ __forceinline__ float round_bf16(float v) { return bf16_bits_to_f32(f32_to_bf16_bits(v)); }

__global__ __launch_bounds__(256) void conv_dense_kernel(const DenseConvArgs a) {
    __shared__ __attribute__((aligned(16))) float wl[kDenseChunk * kDenseFilters];
    const int64_t M = (int64_t)a.N * a.P * a.Q;
    const int n = a.R * a.S * a.C;
    const int k0 = blockIdx.y * kDenseFilters;
    const int64_t m = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const bool live = m < M;

    int h0 = 0, w0 = 0;
    int64_t xbase = 0;
    if (live) {
        const int64_t PQ = (int64_t)a.P * a.Q;
        const int64_t img = m / PQ;
        const int pq = (int)(m - img * PQ);
        const int p = pq / a.Q, q = pq - (pq / a.Q) * a.Q;
        h0 = p * a.sh - a.ph;
        w0 = q * a.sw - a.pw;
        xbase = ((img * a.H + h0) * a.W + w0) * (int64_t)a.C;
    }
    float acc[kDenseFilters];
#pragma unroll
    for (int j = 0; j < kDenseFilters; ++j) acc[j] = 0.0f;

    // (r, s, c) of the next reduction element, carried across LDS fills
    int r = 0, s = 0, c = 0;
    for (int i0 = 0; i0 < n; i0 += kDenseChunk) {
        const int len = min(kDenseChunk, n - i0);
        __syncthreads();  // the previous fill is consumed
        for (int e = threadIdx.x; e < len * kDenseFilters; e += 256) {
            const int j = e % kDenseFilters, i = e / kDenseFilters;
            const int k = k0 + j;
            wl[e] = k < a.K ? round_bf16(a.w[(int64_t)k * n + i0 + i]) : 0.0f;
        }
        __syncthreads();
        if (live) {
            for (int i = 0; i < len; ++i) {
                const int h = h0 + r, w = w0 + s;
                if ((unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W) {
                    const int64_t xi = xbase + ((int64_t)r * a.W + s) * a.C + c;
                    const float xv = a.x_f32 ? round_bf16(reinterpret_cast<const float*>(a.x)[xi])
                                             : bf16_bits_to_f32(reinterpret_cast<const uint16_t*>(a.x)[xi]);
                    const f32x4* wp = reinterpret_cast<const f32x4*>(&wl[i * kDenseFilters]);
#pragma unroll
                    for (int v = 0; v < kDenseFilters / 4; ++v) {
                        const f32x4 w4 = wp[v];
                        acc[4 * v] = fmaf(xv, w4.x, acc[4 * v]);
                        acc[4 * v + 1] = fmaf(xv, w4.y, acc[4 * v + 1]);
                        acc[4 * v + 2] = fmaf(xv, w4.z, acc[4 * v + 2]);
                        acc[4 * v + 3] = fmaf(xv, w4.w, acc[4 * v + 3]);
                    }
                }
                if (++c == a.C) {
                    c = 0;
                    if (++s == a.S) {
                        s = 0;
                        ++r;
                    }
                }
            }
        }
    }
    if (!live) return;

    // epilogue: y = act(acc * scale + bias + residual)
    const int64_t o = m * a.K + k0;
#pragma unroll
    for (int j = 0; j < kDenseFilters; ++j) {
        const int k = k0 + j;
        if (k >= a.K) break;
        float v = acc[j];
        if (a.scale) v *= a.scale[k];
        if (a.bias) v += a.bias[k];
        if (a.residual)
            v += a.y_f32 ? reinterpret_cast<const float*>(a.residual)[o + j]
                         : bf16_bits_to_f32(reinterpret_cast<const uint16_t*>(a.residual)[o + j]);
        if (a.relu) v = fmaxf(v, 0.0f);
        acc[j] = v;
    }
    const bool full = k0 + kDenseFilters <= a.K && a.K % 8 == 0;
    if (a.y_f32) {
        float* yp = reinterpret_cast<float*>(a.y) + o;
        if (full) {
#pragma unroll
            for (int v = 0; v < kDenseFilters / 4; ++v)
                *reinterpret_cast<f32x4*>(yp + 4 * v) = f32x4{acc[4 * v], acc[4 * v + 1], acc[4 * v + 2], acc[4 * v + 3]};
        } else {
            for (int j = 0; j < kDenseFilters && k0 + j < a.K; ++j) yp[j] = acc[j];
        }
    } else {
        uint16_t* yp = reinterpret_cast<uint16_t*>(a.y) + o;
        if (full) {
#pragma unroll
            for (int v = 0; v < kDenseFilters / 8; ++v)
                *reinterpret_cast<u32x4*>(yp + 8 * v) =
                    u32x4{pack_bf16x2(acc[8 * v], acc[8 * v + 1]), pack_bf16x2(acc[8 * v + 2], acc[8 * v + 3]),
                          pack_bf16x2(acc[8 * v + 4], acc[8 * v + 5]), pack_bf16x2(acc[8 * v + 6], acc[8 * v + 7])};
        } else {
            for (int j = 0; j < kDenseFilters && k0 + j < a.K; ++j) yp[j] = (uint16_t)f32_to_bf16_bits(acc[j]);
        }
    }
}

}  // namespace

hipError_t launch_conv_dense(const DenseConvArgs& a, hipStream_t stream) {
    const int64_t M = (int64_t)a.N * a.P * a.Q;
    const dim3 grid((unsigned)((M + 255) / 256), (unsigned)((a.K + kDenseFilters - 1) / kDenseFilters));
    hipLaunchKernelGGL(conv_dense_kernel, grid, dim3(256), 0, stream, a);
    return hipGetLastError();
}

}  // namespace tbn
