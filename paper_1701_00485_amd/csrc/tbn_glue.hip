// tbn_glue.hip -- the layers the workloads put around the two-bit convolutions
// (Sec. 4 uses ResNet-18 with batch normalisation; the smaller workloads add max pooling,
// ReLU and a softmax cross-entropy loss).  All HBM-bound, NHWC bf16 activations.
//   * max pooling forward (argmax kept for the backward pass; ties go to the first
//     maximum in row-major window order) and backward (gather, deterministic);
//   * global average pooling;
//   * batch normalisation in training form (batch statistics) forward and backward,
//     with ReLU fused on both sides;
//   * softmax cross-entropy over fp32 logits (loss and gradient).
#include "tbn_device.h"
#include "tbn_kernels.h"

namespace tbn {

namespace {

__device__ __forceinline__ void st_act(void* p, int64_t i, float v, int f32) {
    if (f32)
        reinterpret_cast<float*>(p)[i] = v;
    else
        reinterpret_cast<uint16_t*>(p)[i] = (uint16_t)f32_to_bf16_bits(v);
}

__global__ __launch_bounds__(256) void maxpool_fwd_kernel(const PoolArgs a, const uint16_t* __restrict__ x,
                                                          uint16_t* __restrict__ y, int32_t* __restrict__ arg) {
    const int64_t total = (int64_t)a.N * a.P * a.Q * a.C;
    const int64_t o = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (o >= total) return;
    const int c = (int)(o % a.C);
    const int64_t pix = o / a.C;
    const int q = (int)(pix % a.Q), p = (int)((pix / a.Q) % a.P);
    const int64_t n = pix / ((int64_t)a.P * a.Q);
    float best = 0.0f;
    int bi = -1;
    for (int r = 0; r < a.k; ++r) {
        const int h = p * a.s - a.pad + r;
        if ((unsigned)h >= (unsigned)a.H) continue;
        for (int t = 0; t < a.k; ++t) {
            const int w = q * a.s - a.pad + t;
            if ((unsigned)w >= (unsigned)a.W) continue;
            const float v = bf16_bits_to_f32(x[((n * a.H + h) * a.W + w) * a.C + c]);
            if (bi < 0 || v > best) {
                best = v;
                bi = h * a.W + w;
            }
        }
    }
    y[o] = (uint16_t)f32_to_bf16_bits(best);  // exact: the maximum is a bf16 value
    if (arg) arg[o] = bi;
}

// dx[n,h,w,c] = sum of dy over the windows that chose (h, w)
__global__ __launch_bounds__(256) void maxpool_bwd_kernel(const PoolArgs a, const uint16_t* __restrict__ dy,
                                                          const int32_t* __restrict__ arg, void* __restrict__ dx,
                                                          int dx_f32) {
    const int64_t total = (int64_t)a.N * a.H * a.W * a.C;
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= total) return;
    const int c = (int)(i % a.C);
    const int64_t pix = i / a.C;
    const int w = (int)(pix % a.W), h = (int)((pix / a.W) % a.H);
    const int64_t n = pix / ((int64_t)a.H * a.W);
    const int me = h * a.W + w;
    // windows p with p*s - pad <= h <= p*s - pad + k - 1
    const int p_lo = max(0, (h + a.pad - a.k + a.s) / a.s), p_hi = min(a.P - 1, (h + a.pad) / a.s);
    const int q_lo = max(0, (w + a.pad - a.k + a.s) / a.s), q_hi = min(a.Q - 1, (w + a.pad) / a.s);
    float acc = 0.0f;
    for (int p = p_lo; p <= p_hi; ++p)
        for (int q = q_lo; q <= q_hi; ++q) {
            const int64_t o = ((n * a.P + p) * a.Q + q) * a.C + c;
            if (arg[o] == me) acc += bf16_bits_to_f32(dy[o]);
        }
    st_act(dx, i, acc, dx_f32);
}

// y[n][c] = mean over h, w of x[n][h][w][c]; one thread per (n, c)
__global__ __launch_bounds__(256) void avgpool_kernel(int32_t N, int32_t HW, int32_t C, const uint16_t* __restrict__ x,
                                                      void* __restrict__ y, int y_f32) {
    const int64_t o = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (o >= (int64_t)N * C) return;
    const int c = (int)(o % C);
    const int64_t n = o / C;
    float acc = 0.0f;
    for (int i = 0; i < HW; ++i) acc += bf16_bits_to_f32(x[(n * HW + i) * C + c]);
    st_act(y, o, acc / (float)HW, y_f32);
}

// ---- batch normalisation, training form ----
// Per-channel statistics over rows = N*H*W: a block of 256 threads owns 8 channels
// (one 16-byte column strip), 32 row groups accumulate in fp32 and combine in LDS; the
// result is written as (mean, inv_std).  Deterministic (fixed reduction order).
__global__ __launch_bounds__(256) void bn_stats_kernel(const uint16_t* __restrict__ x, int64_t rows, int32_t C,
                                                       float eps, float* __restrict__ mean,
                                                       float* __restrict__ inv_std) {
    __shared__ float s1[32][8], s2[32][8];
    const int cl = threadIdx.x & 7, rg = threadIdx.x >> 3;
    const int c = blockIdx.x * 8 + cl;
    float a1 = 0.0f;
    if (c < C)
        for (int64_t r = rg; r < rows; r += 32) a1 += bf16_bits_to_f32(x[r * C + c]);
    s1[rg][cl] = a1;
    __syncthreads();
    if (rg == 0) {
        float t = 0.0f;
        for (int g = 0; g < 32; ++g) t += s1[g][cl];
        s1[0][cl] = t / (float)rows;
    }
    __syncthreads();
    const float m = s1[0][cl];
    float a2 = 0.0f;
    if (c < C)
        for (int64_t r = rg; r < rows; r += 32) {
            const float d = bf16_bits_to_f32(x[r * C + c]) - m;
            a2 += d * d;
        }
    s2[rg][cl] = a2;
    __syncthreads();
    if (rg == 0 && c < C) {
        float t = 0.0f;
        for (int g = 0; g < 32; ++g) t += s2[g][cl];
        mean[c] = m;
        inv_std[c] = 1.0f / sqrtf(t / (float)rows + eps);
    }
}

// y = act(gamma * (x - mean) * inv_std + beta)
__global__ __launch_bounds__(256) void bn_apply_kernel(const uint16_t* __restrict__ x, int64_t total, int32_t C,
                                                       const float* __restrict__ mean, const float* __restrict__ inv_std,
                                                       const float* __restrict__ gamma, const float* __restrict__ beta,
                                                       int relu, uint16_t* __restrict__ y) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= total) return;
    const int c = (int)(i % C);
    float v = gamma[c] * (bf16_bits_to_f32(x[i]) - mean[c]) * inv_std[c] + beta[c];
    if (relu) v = fmaxf(v, 0.0f);
    y[i] = (uint16_t)f32_to_bf16_bits(v);
}

// Backward: g = dy * [y > 0] (when relu), then per channel sums of g and g * xhat.
__global__ __launch_bounds__(256) void bn_bwd_stats_kernel(const uint16_t* __restrict__ x, const uint16_t* __restrict__ y,
                                                           const uint16_t* __restrict__ dy, int64_t rows, int32_t C,
                                                           int relu, const float* __restrict__ mean,
                                                           const float* __restrict__ inv_std, float* __restrict__ dgamma,
                                                           float* __restrict__ dbeta) {
    __shared__ float s1[32][8], s2[32][8];
    const int cl = threadIdx.x & 7, rg = threadIdx.x >> 3;
    const int c = blockIdx.x * 8 + cl;
    float a1 = 0.0f, a2 = 0.0f;
    if (c < C) {
        const float m = mean[c], is = inv_std[c];
        for (int64_t r = rg; r < rows; r += 32) {
            const int64_t i = r * C + c;
            float g = bf16_bits_to_f32(dy[i]);
            if (relu && !(bf16_bits_to_f32(y[i]) > 0.0f)) g = 0.0f;
            a1 += g;
            a2 += g * (bf16_bits_to_f32(x[i]) - m) * is;
        }
    }
    s1[rg][cl] = a1;
    s2[rg][cl] = a2;
    __syncthreads();
    if (rg == 0 && c < C) {
        float t1 = 0.0f, t2 = 0.0f;
        for (int g = 0; g < 32; ++g) {
            t1 += s1[g][cl];
            t2 += s2[g][cl];
        }
        dbeta[c] = t1;
        dgamma[c] = t2;
    }
}

// dx = gamma * inv_std * (g - dbeta / rows - xhat * dgamma / rows)
__global__ __launch_bounds__(256) void bn_bwd_apply_kernel(const uint16_t* __restrict__ x, const uint16_t* __restrict__ y,
                                                           const uint16_t* __restrict__ dy, int64_t total, int64_t rows,
                                                           int32_t C, int relu, const float* __restrict__ mean,
                                                           const float* __restrict__ inv_std,
                                                           const float* __restrict__ gamma,
                                                           const float* __restrict__ dgamma,
                                                           const float* __restrict__ dbeta, uint16_t* __restrict__ dx) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= total) return;
    const int c = (int)(i % C);
    float g = bf16_bits_to_f32(dy[i]);
    if (relu && !(bf16_bits_to_f32(y[i]) > 0.0f)) g = 0.0f;
    const float xh = (bf16_bits_to_f32(x[i]) - mean[c]) * inv_std[c];
    const float inv_rows = 1.0f / (float)rows;
    const float v = gamma[c] * inv_std[c] * (g - dbeta[c] * inv_rows - xh * dgamma[c] * inv_rows);
    dx[i] = (uint16_t)f32_to_bf16_bits(v);
}

// gradient of ReLU applied after the fact: g = dy * [y > 0]
__global__ __launch_bounds__(256) void relu_bwd_kernel(const uint16_t* __restrict__ y, const uint16_t* __restrict__ dy,
                                                       int64_t total, uint16_t* __restrict__ dx) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= total) return;
    dx[i] = bf16_bits_to_f32(y[i]) > 0.0f ? dy[i] : (uint16_t)0;
}

// softmax cross-entropy, mean over the batch: one wave per sample (classes <= 64 * 32)
__global__ __launch_bounds__(64) void softmax_xent_kernel(const float* __restrict__ z, const int32_t* __restrict__ labels,
                                                          int32_t N, int32_t K, float* __restrict__ loss_per_sample,
                                                          uint16_t* __restrict__ dz) {
    const int n = blockIdx.x, lane = threadIdx.x;
    const float* zn = z + (int64_t)n * K;
    float mx = -INFINITY;
    for (int j = lane; j < K; j += 64) mx = fmaxf(mx, zn[j]);
    for (int off = 32; off >= 1; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
    float se = 0.0f;
    for (int j = lane; j < K; j += 64) se += expf(zn[j] - mx);
    for (int off = 32; off >= 1; off >>= 1) se += __shfl_xor(se, off, 64);
    const float lse = mx + logf(se);
    const int lab = labels[n];
    for (int j = lane; j < K; j += 64) {
        const float pj = expf(zn[j] - lse);
        dz[(int64_t)n * K + j] = (uint16_t)f32_to_bf16_bits((pj - (j == lab ? 1.0f : 0.0f)) / (float)N);
    }
    if (lane == 0) loss_per_sample[n] = lse - zn[lab];
}

// mean of the per-sample losses, summed in index order by one wave
__global__ __launch_bounds__(64) void mean_kernel(const float* __restrict__ v, int32_t n, float* __restrict__ out) {
    float acc = 0.0f;
    if (threadIdx.x == 0) {
        for (int i = 0; i < n; ++i) acc += v[i];
        *out = acc / (float)n;
    }
}

unsigned blocks_for(int64_t total) { return (unsigned)((total + 255) / 256); }

}  // namespace

hipError_t launch_maxpool_fwd(const PoolArgs& a, const uint16_t* x, uint16_t* y, int32_t* arg, hipStream_t s) {
    hipLaunchKernelGGL(maxpool_fwd_kernel, dim3(blocks_for((int64_t)a.N * a.P * a.Q * a.C)), dim3(256), 0, s, a, x, y,
                       arg);
    return hipGetLastError();
}

hipError_t launch_maxpool_bwd(const PoolArgs& a, const uint16_t* dy, const int32_t* arg, void* dx, int dx_f32,
                              hipStream_t s) {
    hipLaunchKernelGGL(maxpool_bwd_kernel, dim3(blocks_for((int64_t)a.N * a.H * a.W * a.C)), dim3(256), 0, s, a, dy,
                       arg, dx, dx_f32);
    return hipGetLastError();
}

hipError_t launch_avgpool(int32_t N, int32_t HW, int32_t C, const uint16_t* x, void* y, int y_f32, hipStream_t s) {
    hipLaunchKernelGGL(avgpool_kernel, dim3(blocks_for((int64_t)N * C)), dim3(256), 0, s, N, HW, C, x, y, y_f32);
    return hipGetLastError();
}

hipError_t launch_bn_train_fwd(const uint16_t* x, int64_t rows, int32_t C, const float* gamma, const float* beta,
                               float eps, int relu, uint16_t* y, float* mean, float* inv_std, hipStream_t s) {
    hipLaunchKernelGGL(bn_stats_kernel, dim3((unsigned)((C + 7) / 8)), dim3(256), 0, s, x, rows, C, eps, mean, inv_std);
    hipLaunchKernelGGL(bn_apply_kernel, dim3(blocks_for(rows * C)), dim3(256), 0, s, x, rows * C, C, mean, inv_std,
                       gamma, beta, relu, y);
    return hipGetLastError();
}

hipError_t launch_bn_train_bwd(const uint16_t* x, const uint16_t* y, const uint16_t* dy, int64_t rows, int32_t C,
                               int relu, const float* mean, const float* inv_std, const float* gamma, float* dgamma,
                               float* dbeta, uint16_t* dx, hipStream_t s) {
    hipLaunchKernelGGL(bn_bwd_stats_kernel, dim3((unsigned)((C + 7) / 8)), dim3(256), 0, s, x, y, dy, rows, C, relu,
                       mean, inv_std, dgamma, dbeta);
    hipLaunchKernelGGL(bn_bwd_apply_kernel, dim3(blocks_for(rows * C)), dim3(256), 0, s, x, y, dy, rows * C, rows, C,
                       relu, mean, inv_std, gamma, dgamma, dbeta, dx);
    return hipGetLastError();
}

hipError_t launch_relu_bwd(const uint16_t* y, const uint16_t* dy, int64_t total, uint16_t* dx, hipStream_t s) {
    hipLaunchKernelGGL(relu_bwd_kernel, dim3(blocks_for(total)), dim3(256), 0, s, y, dy, total, dx);
    return hipGetLastError();
}

hipError_t launch_softmax_xent(const float* z, const int32_t* labels, int32_t N, int32_t K, float* loss,
                               float* loss_per_sample, uint16_t* dz, hipStream_t s) {
    hipLaunchKernelGGL(softmax_xent_kernel, dim3((unsigned)N), dim3(64), 0, s, z, labels, N, K, loss_per_sample, dz);
    hipLaunchKernelGGL(mean_kernel, dim3(1), dim3(64), 0, s, loss_per_sample, N, loss);
    return hipGetLastError();
}

}  // namespace tbn
