// tbn_wgrad.hip -- gradient with respect to the approximate filter (Algorithm 1, backward
// step), used unchanged as the real-weight gradient (Sec. 3, straight-through):
//     dW[k][j] = sum_m dy[m][k] * x_col[m][j],   m = (n,p,q),  j = (r,s,c),
// a GEMM with a small output (K x R*S*C) and a long reduction over every output pixel.
//
// Work split (256 threads = 4 waves, bf16 MFMA 32x32x16, fp32 accumulation):
//   * grid = (output tiles, reduction splits); split z reduces a contiguous range of
//     64-pixel chunks and writes its fp32 partial tile to the workspace; a second kernel
//     adds the partials in split order, so the result does not depend on scheduling;
//   * both operands arrive with the reduction index outermost in memory (dy is
//     [m][k], x is [n][h][w][c]), so each thread loads a 4-pixel x 8-channel patch
//     (four 16-byte loads, coalesced along channels), transposes it in registers with
//     byte permutes, and writes four 8-byte rows of the pixel-contiguous LDS tile the
//     MFMA operand reads expect;
//   * pixel -> (n, p, q) uses multiply-high division by precomputed constants.
#include "tbn_device.h"
#include "tbn_kernels.h"

namespace tbn {

namespace {

constexpr int BK = 64;
constexpr int LDA = BK + 8;

struct WgradKernelArgs {
    WgradArgs a;
    FastDiv div_q, div_pq;
};

// (lo16 of a, lo16 of b) and (hi16 of a, hi16 of b)
__device__ __forceinline__ uint32_t pack_lo(uint32_t a, uint32_t b) {
    return __builtin_amdgcn_perm(b, a, 0x05040100u);
}
__device__ __forceinline__ uint32_t pack_hi(uint32_t a, uint32_t b) {
    return __builtin_amdgcn_perm(b, a, 0x07060302u);
}

// Writes a 4-row x 8-column bf16 patch (rows = pixels, columns = channels) into a
// pixel-contiguous LDS tile: tile[(col0 + c) * LDA + row0 .. +3] for c = 0..7.
__device__ __forceinline__ void store_transposed(uint16_t* tile, int col0, int row0, const u32x4* r) {
#pragma unroll
    for (int c = 0; c < 8; ++c) {
        const int wi = c >> 1;
        u32x2 v;
        if (c & 1) {
            v.x = pack_hi(r[0][wi], r[1][wi]);
            v.y = pack_hi(r[2][wi], r[3][wi]);
        } else {
            v.x = pack_lo(r[0][wi], r[1][wi]);
            v.y = pack_lo(r[2][wi], r[3][wi]);
        }
        *reinterpret_cast<u32x2*>(&tile[(col0 + c) * LDA + row0]) = v;
    }
}

template <int BM, int BN, int WM, int WN, bool VEC>
__global__ __launch_bounds__(256) void wgrad_kernel(const WgradKernelArgs ka) {
    const WgradArgs& a = ka.a;
    constexpr int WAVES_N = BN / WN;
    static_assert((BM / WM) * (BN / WN) == 4, "four waves per block");
    static_assert(BM == 128 && BN == 128, "staging map assumes 128 x 128 tiles");
    constexpr int TM = WM / 32, TN = WN / 32;

    __shared__ __attribute__((aligned(16))) uint16_t As[2][BM * LDA];  // [k][pixel]
    __shared__ __attribute__((aligned(16))) uint16_t Bs[2][BN * LDA];  // [j][pixel]

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / WAVES_N;
    const int wn = wave % WAVES_N;
    const int half = lane >> 5;
    const int l32 = lane & 31;

    const int K = a.K;
    const int C = a.C;
    const int J = a.R * a.S * C;
    const uint32_t PQ = (uint32_t)a.P * a.Q;
    const int64_t M = (int64_t)a.N * PQ;
    const int64_t nchunks = (M + BK - 1) / BK;
    const int tilesJ = (J + BN - 1) / BN;
    const int tiles = tilesJ * ((K + BM - 1) / BM);
    // XCD-aware order: the blocks one XCD runs are consecutive in (split, tile) order, so
    // the tiles sharing a split's pixel range share that XCD's L2.
    const int t = (int)xcd_remap(blockIdx.x, gridDim.x);
    const int split = t / tiles;
    const int tk = (t % tiles) / tilesJ;
    const int tj = (t % tiles) % tilesJ;
    const int k0 = tk * BM;
    const int j0 = tj * BN;
    const int64_t c_begin = (int64_t)split * a.chunks_per_split;
    int64_t c_end = c_begin + a.chunks_per_split;
    if (c_end > nchunks) c_end = nchunks;

    // staging map: thread -> 4 pixels (pg) x 8 columns (cg).  Pixel groups vary fastest
    // so that the 16 lanes sharing a column write one contiguous 128-byte LDS row segment.
    const int pg = tid & 15;  // pixels 4*pg .. 4*pg+3 of the chunk
    const int cg = tid >> 4;  // columns 8*cg .. 8*cg+7 of the tile
    // dy columns
    const int kcol = k0 + 8 * cg;
    const bool k_ok = kcol < K;
    // x columns: j = (r, s, c) for this thread's 8 channels (VEC: one (r, s) for all 8)
    const int jcol = j0 + 8 * cg;
    const bool j_ok = jcol < J;
    int xr[VEC ? 1 : 8], xs[VEC ? 1 : 8], xc[VEC ? 1 : 8];
#pragma unroll
    for (int e = 0; e < (VEC ? 1 : 8); ++e) {
        const int j = jcol + e;
        xr[e] = 0x40000000;  // outside every image unless j < J
        xs[e] = 0;
        xc[e] = 0;
        if (j < J) {
            const int rs = j / C;
            xc[e] = j - rs * C;
            xr[e] = rs / a.S;
            xs[e] = rs - xr[e] * a.S;
        }
    }
    const uint16_t* __restrict__ dy = a.dy;
    const uint16_t* __restrict__ x = a.x;

    u32x4 ra[4], rb[4];
    auto load = [&](int64_t chunk) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int64_t m = chunk * BK + 4 * pg + i;
            u32x4 va = {0u, 0u, 0u, 0u}, vb = {0u, 0u, 0u, 0u};
            if (m < M) {
                const uint32_t mm = (uint32_t)m;
                const uint32_t img = fdiv(mm, ka.div_pq);
                const uint32_t pq = mm - img * PQ;
                const uint32_t p = fdiv(pq, ka.div_q);
                const uint32_t q = pq - p * (uint32_t)a.Q;
                const int hb = (int)p * a.sh - a.ph;
                const int wb = (int)q * a.sw - a.pw;
                if constexpr (VEC) {
                    if (k_ok) va = *reinterpret_cast<const u32x4*>(dy + m * K + kcol);
                    const int h = hb + xr[0], w = wb + xs[0];
                    if (j_ok && (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W)
                        vb = *reinterpret_cast<const u32x4*>(
                            x + (((int64_t)img * a.H + h) * a.W + w) * C + xc[0]);
                } else {
                    uint32_t ea[8], eb[8];
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        ea[e] = (kcol + e < K) ? dy[m * K + kcol + e] : 0u;
                        const int h = hb + xr[e], w = wb + xs[e];
                        eb[e] = ((unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W)
                                    ? x[(((int64_t)img * a.H + h) * a.W + w) * C + xc[e]]
                                    : 0u;
                    }
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        va[e] = ea[2 * e] | (ea[2 * e + 1] << 16);
                        vb[e] = eb[2 * e] | (eb[2 * e + 1] << 16);
                    }
                }
            }
            ra[i] = va;
            rb[i] = vb;
        }
    };
    auto store = [&](int buf) {
        store_transposed(As[buf], 8 * cg, 4 * pg, ra);
        store_transposed(Bs[buf], 8 * cg, 4 * pg, rb);
    };

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int t = 0; t < TN; ++t)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][t][v] = 0.0f;

    if (c_begin < c_end) {
        load(c_begin);
        store(0);
        __syncthreads();
        for (int64_t chunk = c_begin; chunk < c_end; ++chunk) {
            const int cur = (int)((chunk - c_begin) & 1);
            const bool more = chunk + 1 < c_end;
            if (more) load(chunk + 1);
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                bf16x8 af[TM], bfr[TN];
#pragma unroll
                for (int i = 0; i < TM; ++i)
                    af[i] = *reinterpret_cast<const bf16x8*>(
                        &As[cur][(wm * WM + 32 * i + l32) * LDA + 16 * u + 8 * half]);
#pragma unroll
                for (int t = 0; t < TN; ++t)
                    bfr[t] = *reinterpret_cast<const bf16x8*>(
                        &Bs[cur][(wn * WN + 32 * t + l32) * LDA + 16 * u + 8 * half]);
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int t = 0; t < TN; ++t) acc[i][t] = mfma32(af[i], bfr[t], acc[i][t]);
            }
            if (more) store(cur ^ 1);
            __syncthreads();
        }
    }

    float* out = a.out + (int64_t)split * K * J;
#pragma unroll
    for (int t = 0; t < TN; ++t) {
        const int col = j0 + wn * WN + 32 * t + l32;
        if (col >= J) continue;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int row = k0 + wm * WM + 32 * i + 8 * (v >> 2) + 4 * half + (v & 3);
                if (row < K) {
                    float* o = out + (int64_t)row * J + col;
                    *o = a.accumulate ? *o + acc[i][t][v] : acc[i][t][v];
                }
            }
    }
}

// partials [splits][stride] (the first `count` of each split are summed)
__global__ __launch_bounds__(256) void split_reduce_kernel(const float* __restrict__ part, int32_t splits,
                                                           int64_t count, int64_t stride, float* __restrict__ dw,
                                                           int32_t accumulate) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= count) return;
    float s = accumulate ? dw[i] : 0.0f;
    // eight partials loaded together, then added in split order
    int z = 0;
    for (; z + 8 <= splits; z += 8) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = part[(int64_t)(z + u) * stride + i];
#pragma unroll
        for (int u = 0; u < 8; ++u) s += v[u];
    }
    for (; z < splits; ++z) s += part[(int64_t)z * stride + i];
    dw[i] = s;
}

// The same sum, four consecutive outputs per thread with 16-byte loads (count and stride
// multiples of 4, 16-byte aligned arrays): a quarter of the load instructions for the
// memory-bound pass over all partials.  Each output adds its partials in split order, as
// above, so the results are identical.
__global__ __launch_bounds__(256) void split_reduce_vec4_kernel(const float* __restrict__ part, int32_t splits,
                                                                int64_t count, int64_t stride, float* __restrict__ dw,
                                                                int32_t accumulate) {
    const int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
    if (i >= count) return;
    f32x4 s = accumulate ? *reinterpret_cast<const f32x4*>(dw + i) : f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    int z = 0;
    for (; z + 8 <= splits; z += 8) {
        f32x4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = *reinterpret_cast<const f32x4*>(part + (int64_t)(z + u) * stride + i);
#pragma unroll
        for (int u = 0; u < 8; ++u) s += v[u];
    }
    for (; z < splits; ++z) s += *reinterpret_cast<const f32x4*>(part + (int64_t)z * stride + i);
    *reinterpret_cast<f32x4*>(dw + i) = s;
}

// Few outputs with many splits (first layers: K x R*S*C of a few thousand): G threads
// per output each add every G-th split, then the G sums are added in group order (fixed,
// so the result is the same on every run).
template <int G>
__global__ __launch_bounds__(256) void split_reduce_groups_kernel(const float* __restrict__ part,
                                                                  int32_t splits, int64_t count, int64_t stride,
                                                                  float* __restrict__ dw, int32_t accumulate) {
    constexpr int OPB = 256 / G;  // outputs per block
    __shared__ float sh[256];
    const int o = threadIdx.x % OPB, g = threadIdx.x / OPB;
    const int64_t i = (int64_t)blockIdx.x * OPB + o;
    float s = 0.0f;
    if (i < count)
        for (int z = g; z < splits; z += G) s += part[(int64_t)z * stride + i];
    sh[threadIdx.x] = s;
    __syncthreads();
    if (g == 0 && i < count) {
        float t = accumulate ? dw[i] : 0.0f;
        for (int gg = 0; gg < G; ++gg) t += sh[gg * OPB + o];
        dw[i] = t;
    }
}

// An NHWC tensor with C channels copied into Cp channels (Cp a multiple of 8, zeros in
// channels C..Cp-1), so that the LDS-DMA kernels (8-channel granularity) apply.  One thread
// per pixel and 8-channel group.
__global__ __launch_bounds__(256) void pad_channels_kernel(const uint16_t* __restrict__ x, int64_t pixels, int32_t C,
                                                           int32_t Cp, uint16_t* __restrict__ xp) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int groups = Cp / 8;
    if (i >= pixels * groups) return;
    const int64_t pix = i / groups;
    const int c0 = (int)(i - pix * groups) * 8;
    uint32_t v[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) v[c] = c0 + c < C ? x[pix * C + c0 + c] : 0u;
    *reinterpret_cast<u32x4*>(xp + pix * Cp + c0) =
        u32x4{v[0] | (v[1] << 16), v[2] | (v[3] << 16), v[4] | (v[5] << 16), v[6] | (v[7] << 16)};
}

// Sum of the split partials of an 8-channel filter gradient [splits][rows][8], keeping
// channels c < C: dw[row][c] (+)= sum_z part[z][row][c], G threads per output adding every
// G-th split, combined in group order (fixed).
template <int G>
__global__ __launch_bounds__(256) void split_reduce_compact_kernel(const float* __restrict__ part, int32_t splits,
                                                                   int64_t rows, int32_t C, float* __restrict__ dw,
                                                                   int32_t accumulate) {
    constexpr int OPB = 256 / G;
    __shared__ float sh[256];
    const int o = threadIdx.x % OPB, g = threadIdx.x / OPB;
    const int64_t i = (int64_t)blockIdx.x * OPB + o;  // output (row, c)
    const int64_t count = rows * C;
    const int64_t src = (i / C) * 8 + i % C;
    float s = 0.0f;
    if (i < count)
        for (int z = g; z < splits; z += G) s += part[(int64_t)z * rows * 8 + src];
    sh[threadIdx.x] = s;
    __syncthreads();
    if (g == 0 && i < count) {
        float t = accumulate ? dw[i] : 0.0f;
        for (int gg = 0; gg < G; ++gg) t += sh[gg * OPB + o];
        dw[i] = t;
    }
}

}  // namespace

hipError_t launch_pad_channels(const uint16_t* x, int64_t pixels, int32_t C, int32_t Cp, uint16_t* xp,
                               hipStream_t stream) {
    const int64_t n = pixels * (Cp / 8);
    hipLaunchKernelGGL(pad_channels_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, x, pixels, C, Cp,
                       xp);
    return hipGetLastError();
}

hipError_t launch_split_reduce_compact(const float* partials, int32_t splits, int64_t rows, int32_t C, float* dw,
                                       int32_t accumulate, hipStream_t stream) {
    const int64_t count = rows * C;
    if (count < 65536 && splits >= 32)
        hipLaunchKernelGGL(split_reduce_compact_kernel<16>, dim3((unsigned)((count + 15) / 16)), dim3(256), 0, stream,
                           partials, splits, rows, C, dw, accumulate);
    else
        hipLaunchKernelGGL(split_reduce_compact_kernel<1>, dim3((unsigned)((count + 255) / 256)), dim3(256), 0, stream,
                           partials, splits, rows, C, dw, accumulate);
    return hipGetLastError();
}

hipError_t launch_wgrad(const WgradArgs& a, hipStream_t stream) {
    if (wgrad_dma_eligible(a)) return launch_wgrad_dma(a, stream);
    const int J = a.R * a.S * a.C;
    const int tiles = ((a.K + 127) / 128) * ((J + 127) / 128);
    WgradKernelArgs ka;
    ka.a = a;
    ka.div_q = make_fastdiv((uint32_t)a.Q);
    ka.div_pq = make_fastdiv((uint32_t)a.P * (uint32_t)a.Q);
    const dim3 grid((unsigned)(tiles * a.splits));
    if (a.K % 8 == 0 && a.C % 8 == 0)
        hipLaunchKernelGGL((wgrad_kernel<128, 128, 64, 64, true>), grid, dim3(256), 0, stream, ka);
    else
        hipLaunchKernelGGL((wgrad_kernel<128, 128, 64, 64, false>), grid, dim3(256), 0, stream, ka);
    return hipGetLastError();
}

hipError_t launch_split_reduce(const float* partials, int32_t splits, int64_t count, int64_t stride, float* dw,
                               int32_t accumulate, hipStream_t stream) {
    if (count < 65536 && splits >= 32) {
        hipLaunchKernelGGL(split_reduce_groups_kernel<16>, dim3((unsigned)((count + 15) / 16)), dim3(256), 0, stream,
                           partials, splits, count, stride, dw, accumulate);
    } else if (count % 4 == 0 && stride % 4 == 0 && (((uintptr_t)partials | (uintptr_t)dw) & 15) == 0) {
        hipLaunchKernelGGL(split_reduce_vec4_kernel, dim3((unsigned)((count / 4 + 255) / 256)), dim3(256), 0, stream,
                           partials, splits, count, stride, dw, accumulate);
    } else {
        hipLaunchKernelGGL(split_reduce_kernel, dim3((unsigned)((count + 255) / 256)), dim3(256), 0, stream,
                           partials, splits, count, stride, dw, accumulate);
    }
    return hipGetLastError();
}

}  // namespace tbn
