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

// NV channels per thread (8 = one 16-byte access when C % 8 == 0).  bf16 values compare
// as their fp32 widening; ties keep the first window position in row-major order.
template <int NV>
__global__ __launch_bounds__(256) void maxpool_fwd_kernel(const PoolArgs a, const uint16_t* __restrict__ x,
                                                          uint16_t* __restrict__ y, int32_t* __restrict__ arg) {
    const int64_t total = (int64_t)a.N * a.P * a.Q * a.C;
    const int64_t o = ((int64_t)blockIdx.x * 256 + threadIdx.x) * NV;
    if (o >= total) return;
    const int c = (int)(o % a.C);
    const int64_t pix = o / a.C;
    const int q = (int)(pix % a.Q), p = (int)((pix / a.Q) % a.P);
    const int64_t n = pix / ((int64_t)a.P * a.Q);
    float best[NV];
    int bi[NV];
#pragma unroll
    for (int e = 0; e < NV; ++e) {
        best[e] = 0.0f;
        bi[e] = -1;
    }
    for (int r = 0; r < a.k; ++r) {
        const int h = p * a.s - a.pad + r;
        if ((unsigned)h >= (unsigned)a.H) continue;
        for (int t = 0; t < a.k; ++t) {
            const int w = q * a.s - a.pad + t;
            if ((unsigned)w >= (unsigned)a.W) continue;
            const int64_t xi = ((n * a.H + h) * a.W + w) * a.C + c;
            uint32_t b[NV];
            if constexpr (NV == 8) {
                const u32x4 v = *reinterpret_cast<const u32x4*>(x + xi);
#pragma unroll
                for (int e = 0; e < 8; ++e) b[e] = (e & 1) ? (v[e / 2] >> 16) : (v[e / 2] & 0xFFFFu);
            } else {
                b[0] = x[xi];
            }
#pragma unroll
            for (int e = 0; e < NV; ++e) {
                const float v = bf16_bits_to_f32(b[e]);
                if (bi[e] < 0 || v > best[e]) {
                    best[e] = v;
                    bi[e] = h * a.W + w;
                }
            }
        }
    }
    // exact: each maximum is a bf16 value
    if constexpr (NV == 8) {
        *reinterpret_cast<u32x4*>(y + o) = u32x4{pack_bf16x2(best[0], best[1]), pack_bf16x2(best[2], best[3]),
                                                  pack_bf16x2(best[4], best[5]), pack_bf16x2(best[6], best[7])};
        if (arg) {
            *reinterpret_cast<u32x4*>(arg + o) = u32x4{(uint32_t)bi[0], (uint32_t)bi[1], (uint32_t)bi[2], (uint32_t)bi[3]};
            *reinterpret_cast<u32x4*>(arg + o + 4) =
                u32x4{(uint32_t)bi[4], (uint32_t)bi[5], (uint32_t)bi[6], (uint32_t)bi[7]};
        }
    } else {
        y[o] = (uint16_t)f32_to_bf16_bits(best[0]);
        if (arg) arg[o] = bi[0];
    }
}

// The same for a compile-time K x K window, 8 channels per thread (C % 8 == 0) and 32-bit
// indices (the host checks the sizes): the K*K 16-byte loads of a thread are all issued
// before the first comparison, and the pixel index is split with multiply-shift divisions.
template <int K>
__global__ __launch_bounds__(256) void maxpool_fwd8_kernel(const PoolArgs a, const FastDiv div_g, const FastDiv div_q,
                                                           const FastDiv div_p, const uint32_t groups,
                                                           const uint16_t* __restrict__ x, uint16_t* __restrict__ y,
                                                           int32_t* __restrict__ arg) {
    const uint32_t gi = blockIdx.x * 256u + threadIdx.x;  // (output pixel, 8-channel group)
    if (gi >= groups) return;
    const uint32_t pix = fdiv(gi, div_g);
    const uint32_t c = (gi - pix * (uint32_t)(a.C / 8)) * 8u;
    const uint32_t nq = fdiv(pix, div_q);
    const int q = (int)(pix - nq * (uint32_t)a.Q);
    const uint32_t n = fdiv(nq, div_p);
    const int p = (int)(nq - n * (uint32_t)a.P);
    const int h0 = p * a.s - a.pad, w0 = q * a.s - a.pad;
    u32x4 v[K * K];
    bool ok[K * K];
#pragma unroll
    for (int r = 0; r < K; ++r)
#pragma unroll
        for (int t = 0; t < K; ++t) {
            const int h = h0 + r, w = w0 + t;
            ok[r * K + t] = (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W;
            const uint32_t xi = (((n * (uint32_t)a.H + (uint32_t)h) * (uint32_t)a.W + (uint32_t)w) * (uint32_t)a.C + c);
            v[r * K + t] = ok[r * K + t] ? *reinterpret_cast<const u32x4*>(x + xi) : u32x4{0u, 0u, 0u, 0u};
        }
    float best[8];
    int bi[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        best[e] = 0.0f;
        bi[e] = -1;
    }
#pragma unroll
    for (int j = 0; j < K * K; ++j) {
        if (!ok[j]) continue;
        const int pos = (h0 + j / K) * a.W + (w0 + j % K);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const float f = bf16_bits_to_f32((e & 1) ? (v[j][e / 2] >> 16) : (v[j][e / 2] & 0xFFFFu));
            if (bi[e] < 0 || f > best[e]) {
                best[e] = f;
                bi[e] = pos;
            }
        }
    }
    const uint32_t o = gi * 8u;
    *reinterpret_cast<u32x4*>(y + o) = u32x4{pack_bf16x2(best[0], best[1]), pack_bf16x2(best[2], best[3]),
                                              pack_bf16x2(best[4], best[5]), pack_bf16x2(best[6], best[7])};
    if (arg) {
        *reinterpret_cast<u32x4*>(arg + o) = u32x4{(uint32_t)bi[0], (uint32_t)bi[1], (uint32_t)bi[2], (uint32_t)bi[3]};
        *reinterpret_cast<u32x4*>(arg + o + 4) = u32x4{(uint32_t)bi[4], (uint32_t)bi[5], (uint32_t)bi[6], (uint32_t)bi[7]};
    }
}

// dx[n,h,w,c] = sum of dy over the windows that chose (h, w); NV channels per thread
template <int NV>
__global__ __launch_bounds__(256) void maxpool_bwd_kernel(const PoolArgs a, const uint16_t* __restrict__ dy,
                                                          const int32_t* __restrict__ arg, void* __restrict__ dx,
                                                          int dx_f32) {
    const int64_t total = (int64_t)a.N * a.H * a.W * a.C;
    const int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * NV;
    if (i >= total) return;
    const int c = (int)(i % a.C);
    const int64_t pix = i / a.C;
    const int w = (int)(pix % a.W), h = (int)((pix / a.W) % a.H);
    const int64_t n = pix / ((int64_t)a.H * a.W);
    const int me = h * a.W + w;
    // windows p with p*s - pad <= h <= p*s - pad + k - 1
    const int p_lo = max(0, (h + a.pad - a.k + a.s) / a.s), p_hi = min(a.P - 1, (h + a.pad) / a.s);
    const int q_lo = max(0, (w + a.pad - a.k + a.s) / a.s), q_hi = min(a.Q - 1, (w + a.pad) / a.s);
    float acc[NV];
#pragma unroll
    for (int e = 0; e < NV; ++e) acc[e] = 0.0f;
    for (int p = p_lo; p <= p_hi; ++p)
        for (int q = q_lo; q <= q_hi; ++q) {
            const int64_t o = ((n * a.P + p) * a.Q + q) * a.C + c;
            if constexpr (NV == 8) {
                const u32x4 a0 = *reinterpret_cast<const u32x4*>(arg + o);
                const u32x4 a1 = *reinterpret_cast<const u32x4*>(arg + o + 4);
                const u32x4 d = *reinterpret_cast<const u32x4*>(dy + o);
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const uint32_t ae = e < 4 ? a0[e] : a1[e - 4];
                    const uint32_t db = (e & 1) ? (d[e / 2] >> 16) : (d[e / 2] & 0xFFFFu);
                    if ((int)ae == me) acc[e] += bf16_bits_to_f32(db);
                }
            } else {
                if (arg[o] == me) acc[0] += bf16_bits_to_f32(dy[o]);
            }
        }
    if constexpr (NV == 8) {
        if (dx_f32) {
            float* dp = reinterpret_cast<float*>(dx) + i;
            *reinterpret_cast<f32x4*>(dp) = f32x4{acc[0], acc[1], acc[2], acc[3]};
            *reinterpret_cast<f32x4*>(dp + 4) = f32x4{acc[4], acc[5], acc[6], acc[7]};
        } else {
            *reinterpret_cast<u32x4*>(reinterpret_cast<uint16_t*>(dx) + i) =
                u32x4{pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3]), pack_bf16x2(acc[4], acc[5]),
                      pack_bf16x2(acc[6], acc[7])};
        }
    } else {
        st_act(dx, i, acc[0], dx_f32);
    }
}

// The same gather over 8-channel groups with 32-bit multiply-shift index splits (sizes below
// 2^31): the kernel above spends most of its instructions on 64-bit divisions.
__global__ __launch_bounds__(256) void maxpool_bwd8_kernel(const PoolArgs a, const FastDiv div_g, const FastDiv div_w,
                                                           const FastDiv div_h, const uint32_t groups,
                                                           const uint16_t* __restrict__ dy,
                                                           const int32_t* __restrict__ arg, void* __restrict__ dx,
                                                           int dx_f32) {
    const uint32_t gi = blockIdx.x * 256u + threadIdx.x;  // (input pixel, 8-channel group)
    if (gi >= groups) return;
    const uint32_t pix = fdiv(gi, div_g);
    const uint32_t c = (gi - pix * (uint32_t)(a.C / 8)) * 8u;
    const uint32_t nh = fdiv(pix, div_w);
    const int w = (int)(pix - nh * (uint32_t)a.W);
    const uint32_t n = fdiv(nh, div_h);
    const int h = (int)(nh - n * (uint32_t)a.H);
    const int me = h * a.W + w;
    const int p_lo = max(0, (h + a.pad - a.k + a.s) / a.s), p_hi = min(a.P - 1, (h + a.pad) / a.s);
    const int q_lo = max(0, (w + a.pad - a.k + a.s) / a.s), q_hi = min(a.Q - 1, (w + a.pad) / a.s);
    float acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.0f;
    for (int p = p_lo; p <= p_hi; ++p)
        for (int q = q_lo; q <= q_hi; ++q) {
            const uint32_t o = ((n * (uint32_t)a.P + (uint32_t)p) * (uint32_t)a.Q + (uint32_t)q) * (uint32_t)a.C + c;
            const u32x4 a0 = *reinterpret_cast<const u32x4*>(arg + o);
            const u32x4 a1 = *reinterpret_cast<const u32x4*>(arg + o + 4);
            const u32x4 d = *reinterpret_cast<const u32x4*>(dy + o);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const uint32_t ae = e < 4 ? a0[e] : a1[e - 4];
                const uint32_t db = (e & 1) ? (d[e / 2] >> 16) : (d[e / 2] & 0xFFFFu);
                if ((int)ae == me) acc[e] += bf16_bits_to_f32(db);
            }
        }
    const uint32_t i = gi * 8u;
    if (dx_f32) {
        float* dp = reinterpret_cast<float*>(dx) + i;
        *reinterpret_cast<f32x4*>(dp) = f32x4{acc[0], acc[1], acc[2], acc[3]};
        *reinterpret_cast<f32x4*>(dp + 4) = f32x4{acc[4], acc[5], acc[6], acc[7]};
    } else {
        *reinterpret_cast<u32x4*>(reinterpret_cast<uint16_t*>(dx) + i) =
            u32x4{pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3]), pack_bf16x2(acc[4], acc[5]),
                  pack_bf16x2(acc[6], acc[7])};
    }
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

// C % 8 == 0: eight lanes per group of 8 channels of one image; lane j sums positions
// j, j + 8, ... with 16-byte loads, then the eight partial sums are combined by a fixed
// butterfly (the result does not depend on scheduling).
__global__ __launch_bounds__(256) void avgpool8_kernel(int32_t N, int32_t HW, int32_t C, const uint16_t* __restrict__ x,
                                                       void* __restrict__ y, int y_f32) {
    const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t grp = t >> 3;  // (n, channel group), N * C / 8 of them
    const int j = (int)(t & 7);
    const int G = C / 8;
    const bool ok = grp < (int64_t)N * G;
    const int64_t n = ok ? grp / G : 0;
    const int c0 = ok ? (int)(grp - n * G) * 8 : 0;
    float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    if (ok) {
        for (int i = j; i < HW; i += 8) {
            const u32x4 v = *reinterpret_cast<const u32x4*>(x + (n * HW + i) * C + c0);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                acc[2 * e] += bf16_bits_to_f32(v[e] & 0xFFFFu);
                acc[2 * e + 1] += bf16_bits_to_f32(v[e] >> 16);
            }
        }
    }
    // every lane of the wave takes part in the shuffles (groups of 8 lanes never straddle
    // a wave; lanes past the end carry zeros)
#pragma unroll
    for (int m = 1; m < 8; m <<= 1)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] += __shfl_xor(acc[e], m, 8);
    if (!ok || j != 0) return;
    const float inv = 1.0f / (float)HW;
    const int64_t o = n * C + c0;
    if (y_f32) {
        float* yp = reinterpret_cast<float*>(y) + o;
        *reinterpret_cast<f32x4*>(yp) = f32x4{acc[0] * inv, acc[1] * inv, acc[2] * inv, acc[3] * inv};
        *reinterpret_cast<f32x4*>(yp + 4) = f32x4{acc[4] * inv, acc[5] * inv, acc[6] * inv, acc[7] * inv};
    } else {
        *reinterpret_cast<u32x4*>(reinterpret_cast<uint16_t*>(y) + o) =
            u32x4{pack_bf16x2(acc[0] * inv, acc[1] * inv), pack_bf16x2(acc[2] * inv, acc[3] * inv),
                  pack_bf16x2(acc[4] * inv, acc[5] * inv), pack_bf16x2(acc[6] * inv, acc[7] * inv)};
    }
}

// ---- batch normalisation, training form ----
// Per-channel sums over rows = N*H*W in two deterministic levels:
//   * partial: block (b, slice) sums rows [b*rpc, (b+1)*rpc) for up to 256 channel groups
//     (8 channels = one 16-byte load per row when C % 8 == 0, else 1); the 256 threads
//     cover tpr = 256 / groups rows at a time, then combine their row lanes through LDS in
//     a fixed order and write partial[b][c];
//   * finalize: one thread per channel adds partial[0..chunks)[c] in order.
// Modes: BN_STATS sums d and d^2 with d = x - x[0][c] (one pass for both statistics: the
// first row's value of each channel is a shift common to every chunk, so the chunk sums
// add, and the variance S2/n - (S1/n)^2 of the shifted values does not cancel against a
// large mean); BN_BWD sums g and g * xhat, with g = dy masked by y > 0 when ReLU followed
// the normalisation.
enum { BN_BWD = 2, BN_STATS = 3 };

template <int MODE, bool VEC>
__global__ __launch_bounds__(256) void bn_partial_kernel(const uint16_t* __restrict__ x, const uint16_t* __restrict__ y,
                                                         const uint16_t* __restrict__ dy, int64_t rows, int32_t C,
                                                         int64_t rpc, int relu, const float* __restrict__ mean,
                                                         const float* __restrict__ inv_std, float* __restrict__ p1,
                                                         float* __restrict__ p2) {
    constexpr int NV = VEC ? 8 : 1;
    constexpr bool TWO = MODE == BN_BWD || MODE == BN_STATS;  // two sums per channel
    __shared__ float s1[256 * NV], s2[TWO ? 256 * NV : 1];
    const int G = VEC ? C / 8 : C;
    const int gbase = blockIdx.y * 256;
    const int Gs = min(256, G - gbase);
    const int tpr = 256 / Gs;
    const int t = threadIdx.x;
    const int g = t % Gs, r0 = t / Gs;
    const bool active = r0 < tpr;
    const int c0 = (gbase + g) * NV;
    const int64_t rbeg = (int64_t)blockIdx.x * rpc;
    const int64_t rend = min(rows, rbeg + rpc);
    float a1[NV], a2[NV], m[NV], is[NV];
#pragma unroll
    for (int e = 0; e < NV; ++e) {
        a1[e] = a2[e] = 0.0f;
        m[e] = MODE == BN_BWD ? mean[c0 + e] : 0.0f;
        is[e] = MODE == BN_BWD ? inv_std[c0 + e] : 0.0f;
    }
    if constexpr (MODE == BN_STATS) {
        // the shift: channel c0 + e of row 0
        if constexpr (VEC) {
            const u32x4 kw = *reinterpret_cast<const u32x4*>(x + c0);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                m[2 * e] = bf16_bits_to_f32(kw[e] & 0xFFFFu);
                m[2 * e + 1] = bf16_bits_to_f32(kw[e] >> 16);
            }
        } else {
            m[0] = bf16_bits_to_f32(x[c0]);
        }
    }
    if (active) {
        for (int64_t r = rbeg + r0; r < rend; r += tpr) {
            const int64_t i = r * C + c0;
            float xv[NV], dv[NV], yv[NV];
            if constexpr (VEC) {
                const u32x4 xw = *reinterpret_cast<const u32x4*>(x + i);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    xv[2 * e] = bf16_bits_to_f32(xw[e] & 0xFFFFu);
                    xv[2 * e + 1] = bf16_bits_to_f32(xw[e] >> 16);
                }
                if constexpr (MODE == BN_BWD) {
                    const u32x4 dw = *reinterpret_cast<const u32x4*>(dy + i);
                    const u32x4 yw = *reinterpret_cast<const u32x4*>(y + i);
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        dv[2 * e] = bf16_bits_to_f32(dw[e] & 0xFFFFu);
                        dv[2 * e + 1] = bf16_bits_to_f32(dw[e] >> 16);
                        yv[2 * e] = bf16_bits_to_f32(yw[e] & 0xFFFFu);
                        yv[2 * e + 1] = bf16_bits_to_f32(yw[e] >> 16);
                    }
                }
            } else {
                xv[0] = bf16_bits_to_f32(x[i]);
                if constexpr (MODE == BN_BWD) {
                    dv[0] = bf16_bits_to_f32(dy[i]);
                    yv[0] = bf16_bits_to_f32(y[i]);
                }
            }
#pragma unroll
            for (int e = 0; e < NV; ++e) {
                if constexpr (MODE == BN_STATS) {
                    const float d = xv[e] - m[e];
                    a1[e] += d;
                    a2[e] += d * d;
                } else {
                    const float gv = (relu && !(yv[e] > 0.0f)) ? 0.0f : dv[e];
                    a1[e] += gv;
                    a2[e] += gv * (xv[e] - m[e]) * is[e];
                }
            }
        }
    }
    const int W = Gs * NV;  // channels of this slice
    if (active) {
#pragma unroll
        for (int e = 0; e < NV; ++e) {
            s1[r0 * W + g * NV + e] = a1[e];
            if constexpr (TWO) s2[r0 * W + g * NV + e] = a2[e];
        }
    }
    __syncthreads();
    for (int c = t; c < W; c += 256) {
        float u1 = 0.0f, u2 = 0.0f;
        for (int rr = 0; rr < tpr; ++rr) {
            u1 += s1[rr * W + c];
            if constexpr (TWO) u2 += s2[rr * W + c];
        }
        const int64_t o = (int64_t)blockIdx.x * C + gbase * NV + c;
        p1[o] = u1;
        if constexpr (TWO) p2[o] = u2;
    }
}

// Backward sums dbeta = sum g and dgamma = sum g * xhat: 16 channels x 16 chunk lanes per
// block, lane j sums chunks j, j + 16, ... in order, then the 16 lane sums in lane order.
__global__ __launch_bounds__(256) void bn_bwd_finalize_kernel(const float* __restrict__ p1, const float* __restrict__ p2,
                                                              int64_t chunks, int32_t C, float* __restrict__ out1,
                                                              float* __restrict__ out2) {
    __shared__ float s1[16][17], s2[16][17];
    const int cl = threadIdx.x & 15, part = threadIdx.x >> 4;
    const int c = blockIdx.x * 16 + cl;
    float u1 = 0.0f, u2 = 0.0f;
    if (c < C) {
        int64_t b = part;
        for (; b + 48 < chunks; b += 64) {  // four loads in flight, added in chunk order
            const float v0 = p1[b * C + c], v1 = p1[(b + 16) * C + c];
            const float v2 = p1[(b + 32) * C + c], v3 = p1[(b + 48) * C + c];
            u1 += v0;
            u1 += v1;
            u1 += v2;
            u1 += v3;
            {
                const float w0 = p2[b * C + c], w1 = p2[(b + 16) * C + c];
                const float w2 = p2[(b + 32) * C + c], w3 = p2[(b + 48) * C + c];
                u2 += w0;
                u2 += w1;
                u2 += w2;
                u2 += w3;
            }
        }
        for (; b < chunks; b += 16) {
            u1 += p1[b * C + c];
            u2 += p2[b * C + c];
        }
    }
    s1[part][cl] = u1;
    s2[part][cl] = u2;
    __syncthreads();
    if (part != 0 || c >= C) return;
    float t1 = 0.0f, t2 = 0.0f;
    for (int j = 0; j < 16; ++j) {
        t1 += s1[j][cl];
        t2 += s2[j][cl];
    }
    out1[c] = t1;  // dbeta
    out2[c] = t2;  // dgamma
}

// One-pass statistics: the chunk sums S1 = sum d, S2 = sum d^2 (d = x - x[0][c]) added in
// chunk order in fp64 (16 chunk lanes per channel, then the lanes in order), then
// mean = x[0][c] + S1 / n and inv_std = 1 / sqrt(S2 / n - (S1 / n)^2 + eps) (biased variance,
// clamped at zero).
__global__ __launch_bounds__(256) void bn_stats_finalize_kernel(const float* __restrict__ p1, const float* __restrict__ p2,
                                                                int64_t chunks, int32_t C, int64_t rows, float eps,
                                                                const uint16_t* __restrict__ x, float* __restrict__ mean,
                                                                float* __restrict__ inv_std) {
    __shared__ double s1[16][17], s2[16][17];
    const int cl = threadIdx.x & 15, part = threadIdx.x >> 4;
    const int c = blockIdx.x * 16 + cl;
    double u1 = 0.0, u2 = 0.0;
    if (c < C) {
        int64_t b = part;
        for (; b + 7 * 16 < chunks; b += 8 * 16) {  // eight loads of each in flight, added in chunk order
            float v1[8], v2[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                v1[k] = p1[(b + 16 * k) * C + c];
                v2[k] = p2[(b + 16 * k) * C + c];
            }
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                u1 += (double)v1[k];
                u2 += (double)v2[k];
            }
        }
        for (; b < chunks; b += 16) {
            u1 += (double)p1[b * C + c];
            u2 += (double)p2[b * C + c];
        }
    }
    s1[part][cl] = u1;
    s2[part][cl] = u2;
    __syncthreads();
    if (part != 0 || c >= C) return;
    double t1 = 0.0, t2 = 0.0;
    for (int j = 0; j < 16; ++j) {
        t1 += s1[j][cl];
        t2 += s2[j][cl];
    }
    const double n = (double)rows;
    const double d1 = t1 / n;
    double var = t2 / n - d1 * d1;
    if (var < 0.0) var = 0.0;
    mean[c] = (float)((double)bf16_bits_to_f32(x[c]) + d1);
    inv_std[c] = 1.0f / sqrtf((float)var + eps);
}

// y = act(gamma * (x - mean) * inv_std + beta); VEC: 8 channels (16 bytes) per thread
template <bool VEC>
__global__ __launch_bounds__(256) void bn_apply_kernel(const uint16_t* __restrict__ x, int64_t total, int32_t C,
                                                       const float* __restrict__ mean, const float* __restrict__ inv_std,
                                                       const float* __restrict__ gamma, const float* __restrict__ beta,
                                                       int relu, uint16_t* __restrict__ y) {
    constexpr int NV = VEC ? 8 : 1;
    const int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * NV;
    if (i >= total) return;
    const int c0 = (int)(i % C);
    if constexpr (VEC) {
        const u32x4 xw = *reinterpret_cast<const u32x4*>(x + i);
        float v[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const uint32_t b = (e & 1) ? (xw[e / 2] >> 16) : (xw[e / 2] & 0xFFFFu);
            v[e] = gamma[c0 + e] * (bf16_bits_to_f32(b) - mean[c0 + e]) * inv_std[c0 + e] + beta[c0 + e];
            if (relu) v[e] = fmaxf(v[e], 0.0f);
        }
        *reinterpret_cast<u32x4*>(y + i) = u32x4{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]),
                                                  pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7])};
    } else {
        float v = gamma[c0] * (bf16_bits_to_f32(x[i]) - mean[c0]) * inv_std[c0] + beta[c0];
        if (relu) v = fmaxf(v, 0.0f);
        y[i] = (uint16_t)f32_to_bf16_bits(v);
    }
}

// dx = gamma * inv_std * (g - dbeta / rows - xhat * dgamma / rows)
template <bool VEC>
__global__ __launch_bounds__(256) void bn_bwd_apply_kernel(const uint16_t* __restrict__ x, const uint16_t* __restrict__ y,
                                                           const uint16_t* __restrict__ dy, int64_t total, int64_t rows,
                                                           int32_t C, int relu, const float* __restrict__ mean,
                                                           const float* __restrict__ inv_std,
                                                           const float* __restrict__ gamma,
                                                           const float* __restrict__ dgamma,
                                                           const float* __restrict__ dbeta, uint16_t* __restrict__ dx) {
    constexpr int NV = VEC ? 8 : 1;
    const int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * NV;
    if (i >= total) return;
    const int c0 = (int)(i % C);
    const float inv_rows = 1.0f / (float)rows;
    uint32_t xb[NV], yb[NV], db[NV];
    if constexpr (VEC) {
        const u32x4 xw = *reinterpret_cast<const u32x4*>(x + i);
        const u32x4 yw = *reinterpret_cast<const u32x4*>(y + i);
        const u32x4 dw = *reinterpret_cast<const u32x4*>(dy + i);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int sh = (e & 1) * 16;
            xb[e] = (xw[e / 2] >> sh) & 0xFFFFu;
            yb[e] = (yw[e / 2] >> sh) & 0xFFFFu;
            db[e] = (dw[e / 2] >> sh) & 0xFFFFu;
        }
    } else {
        xb[0] = x[i];
        yb[0] = y[i];
        db[0] = dy[i];
    }
    float v[NV];
#pragma unroll
    for (int e = 0; e < NV; ++e) {
        const int c = c0 + e;
        float g = bf16_bits_to_f32(db[e]);
        if (relu && !(bf16_bits_to_f32(yb[e]) > 0.0f)) g = 0.0f;
        const float xh = (bf16_bits_to_f32(xb[e]) - mean[c]) * inv_std[c];
        v[e] = gamma[c] * inv_std[c] * (g - dbeta[c] * inv_rows - xh * dgamma[c] * inv_rows);
    }
    if constexpr (VEC) {
        *reinterpret_cast<u32x4*>(dx + i) = u32x4{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]),
                                                   pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7])};
    } else {
        dx[i] = (uint16_t)f32_to_bf16_bits(v[0]);
    }
}

// gradient of ReLU applied after the fact: g = dy * [y > 0]
// 8 elements (16 bytes of each tensor) per thread; the last thread takes the ragged tail
// element by element
__global__ __launch_bounds__(256) void relu_bwd_kernel(const uint16_t* __restrict__ y, const uint16_t* __restrict__ dy,
                                                       int64_t total, uint16_t* __restrict__ dx) {
    const int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 8;
    if (i >= total) return;
    if (i + 8 <= total) {
        const u32x4 yv = *reinterpret_cast<const u32x4*>(y + i);
        const u32x4 gv = *reinterpret_cast<const u32x4*>(dy + i);
        u32x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const uint32_t lo = bf16_bits_to_f32(yv[e] & 0xFFFFu) > 0.0f ? (gv[e] & 0xFFFFu) : 0u;
            const uint32_t hi = bf16_bits_to_f32(yv[e] >> 16) > 0.0f ? (gv[e] & 0xFFFF0000u) : 0u;
            o[e] = lo | hi;
        }
        *reinterpret_cast<u32x4*>(dx + i) = o;
    } else {
        for (int64_t j = i; j < total; ++j) dx[j] = bf16_bits_to_f32(y[j]) > 0.0f ? dy[j] : (uint16_t)0;
    }
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
    // a label outside [0, K) selects no logit: its loss is NaN and its gradient has no -1
    // term, so the row is never read out of bounds
    const int lab = labels[n];
    const bool lab_ok = lab >= 0 && lab < K;
    for (int j = lane; j < K; j += 64) {
        const float pj = expf(zn[j] - lse);
        dz[(int64_t)n * K + j] = (uint16_t)f32_to_bf16_bits((pj - (j == lab ? 1.0f : 0.0f)) / (float)N);
    }
    if (lane == 0) loss_per_sample[n] = lab_ok ? lse - zn[lab] : __builtin_nanf("");
}

// mean of the per-sample losses, summed in index order by one thread; the block first
// stages the values in LDS in chunks (parallel, coalesced loads), so that the serial sum
// reads LDS instead of waiting on one global load per element
__global__ __launch_bounds__(256) void mean_kernel(const float* __restrict__ v, int32_t n, float* __restrict__ out) {
    constexpr int kChunk = 4096;
    __shared__ float buf[kChunk];
    float acc = 0.0f;
    for (int base = 0; base < n; base += kChunk) {
        const int len = n - base < kChunk ? n - base : kChunk;
        for (int i = threadIdx.x; i < len; i += 256) buf[i] = v[base + i];
        __syncthreads();
        if (threadIdx.x == 0)
            for (int i = 0; i < len; ++i) acc += buf[i];
        __syncthreads();
    }
    if (threadIdx.x == 0) *out = acc / (float)n;
}

unsigned blocks_for(int64_t total) { return (unsigned)((total + 255) / 256); }

}  // namespace

hipError_t launch_maxpool_fwd(const PoolArgs& a, const uint16_t* x, uint16_t* y, int32_t* arg, hipStream_t s) {
    const int64_t total = (int64_t)a.N * a.P * a.Q * a.C;
    const int64_t in_total = (int64_t)a.N * a.H * a.W * a.C;
    if (a.C % 8 == 0 && (a.k == 2 || a.k == 3) && total < 0x7FFFFFFFll && in_total < 0x7FFFFFFFll) {
        const uint32_t groups = (uint32_t)(total / 8);
        const FastDiv dg = make_fastdiv((uint32_t)(a.C / 8)), dq = make_fastdiv((uint32_t)a.Q),
                      dp = make_fastdiv((uint32_t)a.P);
        if (a.k == 3)
            hipLaunchKernelGGL(maxpool_fwd8_kernel<3>, dim3(blocks_for(groups)), dim3(256), 0, s, a, dg, dq, dp, groups,
                               x, y, arg);
        else
            hipLaunchKernelGGL(maxpool_fwd8_kernel<2>, dim3(blocks_for(groups)), dim3(256), 0, s, a, dg, dq, dp, groups,
                               x, y, arg);
    } else if (a.C % 8 == 0)
        hipLaunchKernelGGL(maxpool_fwd_kernel<8>, dim3(blocks_for(total / 8)), dim3(256), 0, s, a, x, y, arg);
    else
        hipLaunchKernelGGL(maxpool_fwd_kernel<1>, dim3(blocks_for(total)), dim3(256), 0, s, a, x, y, arg);
    return hipGetLastError();
}

hipError_t launch_maxpool_bwd(const PoolArgs& a, const uint16_t* dy, const int32_t* arg, void* dx, int dx_f32,
                              hipStream_t s) {
    const int64_t total = (int64_t)a.N * a.H * a.W * a.C;
    const int64_t out_total = (int64_t)a.N * a.P * a.Q * a.C;
    if (a.C % 8 == 0 && total < 0x7FFFFFFFll && out_total < 0x7FFFFFFFll) {
        const uint32_t groups = (uint32_t)(total / 8);
        hipLaunchKernelGGL(maxpool_bwd8_kernel, dim3(blocks_for(groups)), dim3(256), 0, s, a,
                           make_fastdiv((uint32_t)(a.C / 8)), make_fastdiv((uint32_t)a.W), make_fastdiv((uint32_t)a.H),
                           groups, dy, arg, dx, dx_f32);
    } else if (a.C % 8 == 0)
        hipLaunchKernelGGL(maxpool_bwd_kernel<8>, dim3(blocks_for(total / 8)), dim3(256), 0, s, a, dy, arg, dx, dx_f32);
    else
        hipLaunchKernelGGL(maxpool_bwd_kernel<1>, dim3(blocks_for(total)), dim3(256), 0, s, a, dy, arg, dx, dx_f32);
    return hipGetLastError();
}

hipError_t launch_avgpool(int32_t N, int32_t HW, int32_t C, const uint16_t* x, void* y, int y_f32, hipStream_t s) {
    if (C % 8 == 0)  // 16-byte rows (the caller guarantees 16-byte aligned buffers)
        hipLaunchKernelGGL(avgpool8_kernel, dim3(blocks_for((int64_t)N * C)), dim3(256), 0, s, N, HW, C, x, y, y_f32);
    else
        hipLaunchKernelGGL(avgpool_kernel, dim3(blocks_for((int64_t)N * C)), dim3(256), 0, s, N, HW, C, x, y, y_f32);
    return hipGetLastError();
}

BnPlan plan_bn(int64_t rows, int32_t C) {
    BnPlan p;
    p.vec = C % 8 == 0;
    const int G = p.vec ? C / 8 : C;
    const int gs = G < 256 ? G : 256;
    const int tpr = 256 / gs;
    int64_t rpc = (rows + 511) / 512;             // about 512 row chunks
    if (rpc < 8 * (int64_t)tpr) rpc = 8 * (int64_t)tpr;  // at least 8 rows per thread
    p.rpc = rpc;
    p.chunks = (rows + rpc - 1) / rpc;
    p.slices = (G + 255) / 256;
    p.ws_bytes = (size_t)2 * p.chunks * C * 4;
    return p;
}

namespace {

template <int MODE>
void bn_partial(const BnPlan& p, const uint16_t* x, const uint16_t* y, const uint16_t* dy, int64_t rows, int32_t C,
                int relu, const float* mean, const float* inv_std, float* p1, float* p2, hipStream_t s) {
    const dim3 grid((unsigned)p.chunks, (unsigned)p.slices);
    if (p.vec)
        hipLaunchKernelGGL((bn_partial_kernel<MODE, true>), grid, dim3(256), 0, s, x, y, dy, rows, C, p.rpc, relu, mean,
                           inv_std, p1, p2);
    else
        hipLaunchKernelGGL((bn_partial_kernel<MODE, false>), grid, dim3(256), 0, s, x, y, dy, rows, C, p.rpc, relu,
                           mean, inv_std, p1, p2);
}

}  // namespace

hipError_t launch_bn_train_fwd(const uint16_t* x, int64_t rows, int32_t C, const float* gamma, const float* beta,
                               float eps, int relu, uint16_t* y, float* mean, float* inv_std, float* ws,
                               hipStream_t s) {
    const BnPlan p = plan_bn(rows, C);
    float* p1 = ws;
    float* p2 = ws + p.chunks * C;
    const unsigned cb = (unsigned)((C + 15) / 16);
    // one pass over x for both statistics (shifted sums), then the per-channel finalize
    bn_partial<BN_STATS>(p, x, nullptr, nullptr, rows, C, 0, nullptr, nullptr, p1, p2, s);
    hipLaunchKernelGGL(bn_stats_finalize_kernel, dim3(cb), dim3(256), 0, s, p1, p2, p.chunks, C, rows, eps, x, mean,
                       inv_std);
    const int64_t total = rows * C;
    if (p.vec)
        hipLaunchKernelGGL(bn_apply_kernel<true>, dim3(blocks_for(total / 8)), dim3(256), 0, s, x, total, C, mean,
                           inv_std, gamma, beta, relu, y);
    else
        hipLaunchKernelGGL(bn_apply_kernel<false>, dim3(blocks_for(total)), dim3(256), 0, s, x, total, C, mean, inv_std,
                           gamma, beta, relu, y);
    return hipGetLastError();
}

hipError_t launch_bn_train_bwd(const uint16_t* x, const uint16_t* y, const uint16_t* dy, int64_t rows, int32_t C,
                               int relu, const float* mean, const float* inv_std, const float* gamma, float* dgamma,
                               float* dbeta, uint16_t* dx, float* ws, hipStream_t s) {
    const BnPlan p = plan_bn(rows, C);
    float* p1 = ws;
    float* p2 = ws + p.chunks * C;
    bn_partial<BN_BWD>(p, x, y, dy, rows, C, relu, mean, inv_std, p1, p2, s);
    hipLaunchKernelGGL(bn_bwd_finalize_kernel, dim3((unsigned)((C + 15) / 16)), dim3(256), 0, s, p1, p2, p.chunks, C,
                       dbeta, dgamma);
    const int64_t total = rows * C;
    if (p.vec)
        hipLaunchKernelGGL(bn_bwd_apply_kernel<true>, dim3(blocks_for(total / 8)), dim3(256), 0, s, x, y, dy, total, rows,
                           C, relu, mean, inv_std, gamma, dgamma, dbeta, dx);
    else
        hipLaunchKernelGGL(bn_bwd_apply_kernel<false>, dim3(blocks_for(total)), dim3(256), 0, s, x, y, dy, total, rows,
                           C, relu, mean, inv_std, gamma, dgamma, dbeta, dx);
    return hipGetLastError();
}

hipError_t launch_relu_bwd(const uint16_t* y, const uint16_t* dy, int64_t total, uint16_t* dx, hipStream_t s) {
    hipLaunchKernelGGL(relu_bwd_kernel, dim3(blocks_for((total + 7) / 8)), dim3(256), 0, s, y, dy, total, dx);
    return hipGetLastError();
}

hipError_t launch_softmax_xent(const float* z, const int32_t* labels, int32_t N, int32_t K, float* loss,
                               float* loss_per_sample, uint16_t* dz, hipStream_t s) {
    hipLaunchKernelGGL(softmax_xent_kernel, dim3((unsigned)N), dim3(64), 0, s, z, labels, N, K, loss_per_sample, dz);
    hipLaunchKernelGGL(mean_kernel, dim3(1), dim3(256), 0, s, loss_per_sample, N, loss);
    return hipGetLastError();
}

}  // namespace tbn
