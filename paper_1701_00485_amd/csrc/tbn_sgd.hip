// tbn_sgd.hip -- update of the real weights (Algorithm 1, update step) with the optimiser
// of Sec. 4: SGD with momentum and weight decay.  Element-wise and HBM-bound: 12 bytes
// read and 8 written per weight, moved as 16-byte vectors.
#include "tbn_device.h"
#include "tbn_kernels.h"

namespace tbn {

namespace {

// Explicit fused multiply-adds: the same rounding as the fused update-and-quantise kernel.
__device__ __forceinline__ void sgd_one(float& w, float& v, float g, float lr, float mu, float wd) {
    v = __builtin_fmaf(mu, v, __builtin_fmaf(wd, w, g));
    w = __builtin_fmaf(-lr, v, w);
}

__global__ __launch_bounds__(256) void sgd_kernel(float* __restrict__ w, float* __restrict__ v,
                                                  const float* __restrict__ g, int64_t count, float lr,
                                                  float mu, float wd) {
    const int64_t nvec = count / 4;
    const int64_t stride = (int64_t)gridDim.x * 256;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < nvec; i += stride) {
        f32x4 wv = reinterpret_cast<f32x4*>(w)[i];
        f32x4 vv = reinterpret_cast<f32x4*>(v)[i];
        const f32x4 gv = reinterpret_cast<const f32x4*>(g)[i];
        float w0 = wv.x, w1 = wv.y, w2 = wv.z, w3 = wv.w;
        float v0 = vv.x, v1 = vv.y, v2 = vv.z, v3 = vv.w;
        sgd_one(w0, v0, gv.x, lr, mu, wd);
        sgd_one(w1, v1, gv.y, lr, mu, wd);
        sgd_one(w2, v2, gv.z, lr, mu, wd);
        sgd_one(w3, v3, gv.w, lr, mu, wd);
        reinterpret_cast<f32x4*>(w)[i] = f32x4{w0, w1, w2, w3};
        reinterpret_cast<f32x4*>(v)[i] = f32x4{v0, v1, v2, v3};
    }
    // tail (count % 4 elements) handled by the first threads of block 0
    if (blockIdx.x == 0 && threadIdx.x < (count & 3)) {
        const int64_t i = nvec * 4 + threadIdx.x;
        float wi = w[i], vi = v[i];
        sgd_one(wi, vi, g[i], lr, mu, wd);
        w[i] = wi;
        v[i] = vi;
    }
}

}  // namespace

hipError_t launch_sgd(float* w, float* v, const float* g, int64_t count, float lr, float mu, float wd,
                      hipStream_t stream) {
    const int64_t nvec = count / 4;
    int64_t blocks = (nvec + 255) / 256;
    if (blocks < 1) blocks = 1;
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL(sgd_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, w, v, g, count, lr, mu, wd);
    return hipGetLastError();
}

}  // namespace tbn
