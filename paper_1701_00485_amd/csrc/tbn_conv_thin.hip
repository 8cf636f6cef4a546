// tbn_conv_thin.hip -- forward pass of a two-bit layer (Sec. 2 Eq. 1) whose input has few
// channels (C < 8, or fp32 input with C <= 8): image stems such as the 7x7 stride-2
// convolution over RGB, and single-channel MNIST-shaped layers.  The general implicit GEMM
// gathers such inputs element by element; here the block instead
//   * decodes its 64 filters once into LDS as exact bf16 +-1/+-2, laid out with the
//     channels of every tap padded to a power of two CP and the taps of one filter row
//     (s, c) padded to T (a power of two >= 16) elements, padding weights zero;
//   * stages, per output tile of 4 rows x 32 columns of one image, the input patch the
//     tile reads into LDS with the same channel padding, so that the reduction elements
//     (s, c) of one tap row are contiguous both in the patch and in the filters;
//   * runs v_mfma_f32_32x32x16_bf16 over the reduction (r, t), each wave one output row of
//     32 pixels against the 64 filters (two 32x32 accumulators);
//   * applies alpha (and the optional scale, bias, residual, ReLU) in fp32 and writes
//     16-byte rows through a small per-wave LDS transpose.
// Blocks are persistent over the output tiles, so the filter decode is paid once per block.
// For large inputs (the image stems) a first kernel writes the input once into workspace as
// a zero-bordered copy with the padded channel count, and the patches are then copied from it
// straight into LDS in whole 16-byte pieces (LDS-DMA): no per-element bounds checks or
// address arithmetic remain in the tile loop.
#include "tbn_device.h"
#include "tbn_dma.h"
#include "tbn_kernels.h"

namespace tbn {

namespace {

constexpr int TP = 8;    // output rows per tile (two per wave)
constexpr int TQ = 32;   // output columns per tile (one per lane of an MFMA column)
constexpr int FB = 64;   // filters per block
constexpr int SPITCH = 36;  // fp32 pitch of the epilogue transpose (32 filters + 4)

template <int CP>
__device__ __forceinline__ bf16x8 load8(const uint16_t* p) {
    // 8 consecutive bf16 from LDS; the address is aligned to min(2 * CP, 16) bytes
    if constexpr (CP >= 8) {
        return *reinterpret_cast<const bf16x8*>(p);
    } else if constexpr (CP == 4) {
        const u32x2 lo = *reinterpret_cast<const u32x2*>(p);
        const u32x2 hi = *reinterpret_cast<const u32x2*>(p + 4);
        return as_bf16x8(u32x4{lo.x, lo.y, hi.x, hi.y});
    } else if constexpr (CP == 2) {
        const uint32_t* q = reinterpret_cast<const uint32_t*>(p);
        return as_bf16x8(u32x4{q[0], q[1], q[2], q[3]});
    } else {
        u32x4 v;
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = (uint32_t)p[2 * i] | ((uint32_t)p[2 * i + 1] << 16);
        return as_bf16x8(v);
    }
}

// Input patch of one tile, loaded into registers so that the next tile's loads are in
// flight while the current tile computes.  Thread t takes elements t, t + 256, ... of the
// patch in input order (row, then the W*C elements of the row, contiguous in memory, so the
// loads coalesce).  Where each element sits does not depend on the tile, so it is worked
// out once: desc = LDS element index (16 bits) | patch row (6 bits) | patch column (10 bits),
// 0xFFFFFFFF for none.  A loaded register holds the bf16 value (low half) and the LDS index.
constexpr int kElemsPerThread = 24;

template <int CP, bool X32>
__device__ __forceinline__ uint32_t load_patch(const ConvGemmArgs& a, const uint32_t (&desc)[kElemsPerThread],
                                               uint32_t x_img, int hb, int wb, uint32_t (&pv)[kElemsPerThread]) {
    // branch-free, so that all the loads are issued back to back: an element outside the
    // image (or no element) loads x[0].  The raw values are consumed only when the patch is
    // written to LDS (after the next barrier), so nothing waits for them here; bit i of
    // the returned mask says whether value i is real or must be replaced by zero.
    uint32_t okmask = 0;
#pragma unroll
    for (int i = 0; i < kElemsPerThread; ++i) {
        const uint32_t d = desc[i];
        const int h = hb + (int)((d >> 10) & 63), w = wb + (int)(d & 1023);
        const bool ok = d != 0xFFFFFFFFu && (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W;
        const uint32_t xi = ok ? x_img + ((uint32_t)h * a.W + (uint32_t)w) * a.C + ((d >> 16) & (CP - 1)) : 0u;
        if constexpr (X32)
            pv[i] = __float_as_uint(reinterpret_cast<const float*>(a.x)[xi]);
        else
            pv[i] = reinterpret_cast<const uint16_t*>(a.x)[xi];
        okmask |= (ok ? 1u : 0u) << i;
    }
    return okmask;
}

// The zero-bordered copy of the input: xp[n][h'][w'][c] = x[n][h' - ph][w' - pw][c] inside
// the image and for c < C, else 0 (bf16).  One thread per padded pixel, CP elements each.
template <int CP, bool X32>
__global__ __launch_bounds__(256) void thin_pad_kernel(const ConvGemmArgs a, const ThinGeom g, uint16_t* xp) {
    const int64_t total = (int64_t)a.N * g.Hp * g.Wp;
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= total) return;
    const int64_t hw = (int64_t)g.Hp * g.Wp;
    const int n = (int)(i / hw);
    const int rem = (int)(i - (int64_t)n * hw);
    const int hp = rem / g.Wp, wp = rem - (rem / g.Wp) * g.Wp;
    const int h = hp - a.ph, w = wp - a.pw;
    const bool in = (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W;
    const int64_t src = (((int64_t)n * a.H + h) * a.W + w) * a.C;
    uint32_t v[CP];
#pragma unroll
    for (int c = 0; c < CP; ++c) {
        uint32_t e = 0;
        if (in && c < a.C)
            e = X32 ? f32_to_bf16_bits(reinterpret_cast<const float*>(a.x)[src + c])
                    : reinterpret_cast<const uint16_t*>(a.x)[src + c];
        v[c] = e;
    }
    uint16_t* dst = xp + i * CP;
    if constexpr (CP == 1) {
        dst[0] = (uint16_t)v[0];
    } else if constexpr (CP == 2) {
        *reinterpret_cast<uint32_t*>(dst) = v[0] | (v[1] << 16);
    } else if constexpr (CP == 4) {
        *reinterpret_cast<u32x2*>(dst) = u32x2{v[0] | (v[1] << 16), v[2] | (v[3] << 16)};
    } else {
        *reinterpret_cast<u32x4*>(dst) =
            u32x4{v[0] | (v[1] << 16), v[2] | (v[3] << 16), v[4] | (v[5] << 16), v[6] | (v[7] << 16)};
    }
}

// TT: 16-element reduction steps per filter row (T / 16), so that the reduction loop is
// one flat, unrolled sequence whose operand reads run one step ahead of the MFMAs.
// DMA: patches copied from the zero-bordered workspace copy (a.partial) with LDS-DMA.
template <int CP, bool X32, int TT, bool DMA>
__global__ __launch_bounds__(256) void conv_thin_kernel(const ConvGemmArgs a, const ThinGeom g) {
    extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
    uint16_t* wl = reinterpret_cast<uint16_t*>(lds + g.w_off);  // [FB][WPITCH]
    uint16_t* pl = reinterpret_cast<uint16_t*>(lds + g.p_off);  // [PH][PW][CP]
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int half = lane >> 5;
    const int l32 = lane & 31;
    float* st = reinterpret_cast<float*>(lds + g.s_off) + wave * 32 * SPITCH;

    const int K = a.Kf, C = a.C, R = a.R, S = a.S;
    const int n = R * S * C;
    const int NB = (n + 63) / 64;
    const int k0 = blockIdx.y * FB;

    // tile index -> (image, first output row, first output column), by multiply-shift
    // divisions (the host checks that the tile count fits 31 bits)
    const uint32_t PQt = (uint32_t)g.tiles_p * (uint32_t)g.tiles_q;
    auto origin = [&](int64_t tile, int64_t* img, int* p0, int* q0) {
        const uint32_t t32 = (uint32_t)tile;
        const uint32_t im = fdiv(t32, g.div_pqt);
        const uint32_t rem = t32 - im * PQt;
        const uint32_t tp = fdiv(rem, g.div_tq);
        *img = (int64_t)im;
        *p0 = (int)tp * TP;
        *q0 = (int)(rem - tp * (uint32_t)g.tiles_q) * TQ;
    };
    const uint32_t img_elems = (uint32_t)a.H * a.W * a.C;
    uint32_t desc[kElemsPerThread];
#pragma unroll
    for (int i = 0; i < kElemsPerThread; ++i) {
        const uint32_t e = tid + 256 * i;
        desc[i] = 0xFFFFFFFFu;
        if (!DMA && i < g.ept && e < (uint32_t)g.nelem) {
            const uint32_t row = fdiv(e, g.div_rowlen);
            const uint32_t j = e - row * (uint32_t)g.rowlen;
            const uint32_t cell = fdiv(j, g.div_c);
            const uint32_t c = j - cell * (uint32_t)C;
            desc[i] = ((((row * g.PW) + cell) * CP + c) << 16) | (row << 10) | cell;
        }
    }
    // element-wise patches: the first tile's loads are issued before anything else, so that
    // their latency overlaps the filter decode below (one round trip to memory for both)
    int64_t img = 0;
    int p0 = 0, q0 = 0;
    uint32_t pv0[kElemsPerThread];
    uint32_t okm0 = 0;
    if constexpr (!DMA) {
        if (blockIdx.x < g.ntiles) {
            origin(blockIdx.x, &img, &p0, &q0);
            okm0 = load_patch<CP, X32>(a, desc, (uint32_t)img * img_elems, p0 * a.sh - a.ph, q0 * a.sw - a.pw, pv0);
        }
    }

    // ---- the block's filters into LDS as bf16, zero at padding taps / channels / filters:
    //      the packed codes (NB KiB, contiguous in the blocked layout) decoded to W~, or
    //      the real filters of a full-precision layer rounded to bf16 ----
    uint32_t* cw = reinterpret_cast<uint32_t*>(lds + g.s_off);
    if (a.wdense) {
        // a full-precision layer: its real filters rounded to bf16 (nearest even)
        const int f = tid >> 2;
        const bool fk = k0 + f < K;
        for (int j = tid & 3; j < g.WPITCH; j += 4) {
            uint32_t v = 0;
            if (j < g.RT && fk) {
                const int r = j >> g.logT, t = j & (g.T - 1);
                const int s = t / CP, c = t & (CP - 1);
                if (s < S && c < C) v = f32_to_bf16_bits(a.wdense[(int64_t)(k0 + f) * n + (r * S + s) * C + c]);
            }
            wl[f * g.WPITCH + j] = (uint16_t)v;
        }
    } else {
        {
            const u32x4* src = reinterpret_cast<const u32x4*>(a.codes + (int64_t)blockIdx.y * NB * 256);
            for (int i = tid; i < NB * 64; i += 256) reinterpret_cast<u32x4*>(cw)[i] = src[i];
        }
        __syncthreads();
        const int f = tid >> 2;  // 4 threads per filter row
        const bool fk = k0 + f < K;
        for (int j = tid & 3; j < g.WPITCH; j += 4) {
            uint32_t v = 0;
            if (j < g.RT && fk) {
                const int r = j >> g.logT, t = j & (g.T - 1);
                const int s = t / CP, c = t & (CP - 1);
                if (s < S && c < C) {
                    const int i = (r * S + s) * C + c;
                    const uint32_t w = cw[((i >> 6) * 64 + f) * 4 + ((i & 63) >> 4)];
                    const int jj = (i & 15) >> 1, hh = i & 1;
                    const uint32_t mag = (w >> (16 * hh + jj)) & 1u, sg = (w >> (16 * hh + 8 + jj)) & 1u;
                    v = 0x3F80u + (mag << 7) + (sg << 15);  // bf16 of +-1 / +-2
                }
            }
            wl[f * g.WPITCH + j] = (uint16_t)v;
        }
    }

    // ---- epilogue constants: this lane always writes channels k0 + 32 t + 8 (lane % 4) + 0..7 ----
    float cs[2][8], bi[2][8];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int col = k0 + 32 * t + 8 * (lane & 3) + e;
            const bool ok = col < K;
            float sc = ok && a.colscale ? a.colscale[col] : 1.0f;
            if (ok && a.scale) sc *= a.scale[col];
            cs[t][e] = sc;
            bi[t][e] = ok && a.bias ? a.bias[col] : 0.0f;
        }
    const bool vec_store = (K % 8) == 0;

    // channel-padding slots of the patch stay zero; data elements are rewritten per tile
    if constexpr (!DMA) {
        for (int i = tid; i < 2 * g.pbuf; i += 256) pl[i] = 0;
    }
    __syncthreads();  // zeros (and the decoded filters) in place before the first patch

    // the patch is double buffered in LDS: tile i computes from buffer i % 2 while the
    // loads of tile i + 1 are in flight; their values land in the other buffer at the end
    // of the iteration, so no loaded register is carried across the loop edge
    auto write_patch = [&](uint16_t* buf, const uint32_t (&pv)[kElemsPerThread], uint32_t okmask) {
#pragma unroll
        for (int i = 0; i < kElemsPerThread; ++i) {
            if (desc[i] != 0xFFFFFFFFu) {
                const uint32_t v = X32 ? f32_to_bf16_bits(__uint_as_float(pv[i])) : pv[i];
                buf[desc[i] >> 16] = (uint16_t)(((okmask >> i) & 1u) ? v : 0u);
            }
        }
    };
    // the tile's reduction: wave w computes output rows w and w + 4 of the tile
    auto tile_mfma = [&](const uint16_t* cur, f32x16 (&acc)[2][2]) {
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int v = 0; v < 16; ++v) acc[u][t][v] = 0.0f;
        const uint16_t* abase = cur + ((wave * a.sh) * g.PW + l32 * a.sw) * CP + 8 * half;
        const int arow4 = 4 * a.sh * g.PW * CP;  // patch offset of output row + 4
        const int arowr = g.PW * CP;             // patch offset of filter row r + 1
        const uint16_t* bbase = wl + l32 * g.WPITCH + 8 * half;
        // flat reduction steps j = r * TT + t (16 elements each); the filters are contiguous
        // in j, the patch advances a row every TT steps.  Two operand sets alternate, the
        // reads of step j + 1 issued before the MFMAs of step j (no copies at the loop edge)
        const int J = R * TT;
        bf16x8 xa[2], xb[2], wa[2], wb[2];
        auto rd = [&](int j, int s) {
            const uint16_t* an = abase + (j / TT) * arowr + 16 * (j % TT);
            xa[s] = load8<CP>(an);
            xb[s] = load8<CP>(an + arow4);
            wa[s] = *reinterpret_cast<const bf16x8*>(bbase + 16 * j);
            wb[s] = *reinterpret_cast<const bf16x8*>(bbase + 32 * g.WPITCH + 16 * j);
        };
        auto mm = [&](int s) {
            acc[0][0] = mfma32(wa[s], xa[s], acc[0][0]);
            acc[0][1] = mfma32(wb[s], xa[s], acc[0][1]);
            acc[1][0] = mfma32(wa[s], xb[s], acc[1][0]);
            acc[1][1] = mfma32(wb[s], xb[s], acc[1][1]);
        };
        rd(0, 0);
        int j = 0;
        for (; j + 2 <= J; j += 2) {
            rd(j + 1, 1);
            mm(0);
            if (j + 2 < J) rd(j + 2, 0);
            mm(1);
        }
        if (j < J) mm(0);  // odd step count: the last step's operands are in set 0
    };

    auto tile_epilogue = [&](const f32x16 (&acc)[2][2], int64_t cimg, int cp0, int cq0) {
        // ---- epilogue: lane holds pixel l32 and filters 32 t + 8 g + 4 half + 0..3 ----
#pragma unroll
        for (int ut = 0; ut < 4; ++ut) {
            const int u = ut >> 1, t = ut & 1;
            const int p = cp0 + wave + 4 * u;
#pragma unroll
            for (int gq = 0; gq < 4; ++gq)
                *reinterpret_cast<f32x4*>(&st[l32 * SPITCH + 8 * gq + 4 * half]) =
                    f32x4{acc[u][t][4 * gq], acc[u][t][4 * gq + 1], acc[u][t][4 * gq + 2], acc[u][t][4 * gq + 3]};
            __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
#pragma unroll
            for (int pass = 0; pass < 2; ++pass) {
                const int px = (pass * 64 + lane) >> 2, gi = lane & 3;
                const int q = cq0 + px;
                const int col0 = k0 + 32 * t + 8 * gi;
                if (p >= a.P || q >= a.Q || col0 >= K) continue;
                const f32x4 lo = *reinterpret_cast<const f32x4*>(&st[px * SPITCH + 8 * gi]);
                const f32x4 hi = *reinterpret_cast<const f32x4*>(&st[px * SPITCH + 8 * gi + 4]);
                float v8[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
                const int64_t o = ((cimg * a.P + p) * a.Q + q) * K + col0;
#pragma unroll
                for (int e = 0; e < 8; ++e) v8[e] = v8[e] * cs[t][e] + bi[t][e];
                if (a.residual) {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if (col0 + e < K)
                            v8[e] += a.y_f32 ? reinterpret_cast<const float*>(a.residual)[o + e]
                                             : bf16_bits_to_f32(reinterpret_cast<const uint16_t*>(a.residual)[o + e]);
                }
                if (a.relu) {
#pragma unroll
                    for (int e = 0; e < 8; ++e) v8[e] = fmaxf(v8[e], 0.0f);
                }
                if (a.y_f32) {
                    float* yp = reinterpret_cast<float*>(a.y) + o;
                    if (vec_store) {
                        *reinterpret_cast<f32x4*>(yp) = f32x4{v8[0], v8[1], v8[2], v8[3]};
                        *reinterpret_cast<f32x4*>(yp + 4) = f32x4{v8[4], v8[5], v8[6], v8[7]};
                    } else {
                        for (int e = 0; e < 8 && col0 + e < K; ++e) yp[e] = v8[e];
                    }
                } else {
                    uint16_t* yp = reinterpret_cast<uint16_t*>(a.y) + o;
                    if (vec_store) {
                        *reinterpret_cast<u32x4*>(yp) = u32x4{pack_bf16x2(v8[0], v8[1]), pack_bf16x2(v8[2], v8[3]),
                                                             pack_bf16x2(v8[4], v8[5]), pack_bf16x2(v8[6], v8[7])};
                    } else {
                        for (int e = 0; e < 8 && col0 + e < K; ++e) yp[e] = (uint16_t)f32_to_bf16_bits(v8[e]);
                    }
                }
            }
        }
    };

    if constexpr (DMA) {
        // byte offsets, relative to the patch origin in the zero-bordered copy, of the pieces
        // this lane copies: piece k = 64 (4 i + wave) + lane of the patch is row k / ppr,
        // 16-byte column k % ppr, and lands at LDS byte 16 k of the patch buffer (pieces past
        // the patch get an out-of-range offset and land as zeros in the buffer's tail)
        constexpr int kMaxNi = 8;
        uint32_t prel[kMaxNi];
#pragma unroll
        for (int i = 0; i < kMaxNi; ++i) {
            const int k = 64 * (4 * i + wave) + lane;
            const int r = k / g.ppr, j = k - (k / g.ppr) * g.ppr;
            prel[i] = (i < g.ni && k < g.npieces) ? (uint32_t)((r * g.Wp * CP + 8 * j) * 2) : 0x80000000u;
        }
        const v4i rs_xp = make_rsrc(a.partial, (uint32_t)g.ws_bytes);
        auto issue_patch = [&](int64_t t, uint16_t* buf) {
            int64_t im;
            int tp0, tq0;
            origin(t, &im, &tp0, &tq0);
            const uint32_t toff = (uint32_t)((((int64_t)im * g.Hp + (int64_t)tp0 * a.sh) * g.Wp + (int64_t)tq0 * a.sw) * CP * 2);
            const uint32_t base = lds_addr(buf);
#pragma unroll
            for (int i = 0; i < kMaxNi; ++i) {
                if (i < g.ni)
                    dma_b128(rs_xp, base + (uint32_t)(64 * (4 * i + wave)) * 16u,
                             prel[i] >= 0x80000000u ? 0x80000000u : prel[i] + toff);
            }
        };
        int64_t tile = blockIdx.x;
        if (tile < g.ntiles) issue_patch(tile, pl);
        wait_vmcnt(0);
        __syncthreads();
        for (int it = 0; tile < g.ntiles; tile += gridDim.x, ++it) {
            uint16_t* cur = pl + (it & 1) * g.pbuf;
            uint16_t* nxt = pl + ((it + 1) & 1) * g.pbuf;
            int64_t cimg;
            int cp0, cq0;
            origin(tile, &cimg, &cp0, &cq0);
            const bool more = tile + gridDim.x < g.ntiles;
            // the next tile's patch is copied into the other buffer while this one computes
            if (more) issue_patch(tile + gridDim.x, nxt);
            f32x16 acc[2][2];
            tile_mfma(cur, acc);
            // this wave's pieces of the next patch have landed (and the previous tile's
            // stores, issued a whole reduction ago, are done)
            wait_vmcnt(0);
            tile_epilogue(acc, cimg, cp0, cq0);
            __syncthreads();  // the next patch is complete; every wave is done with this one
        }
        return;
    }
    int64_t tile = blockIdx.x;
    if (tile < g.ntiles) write_patch(pl, pv0, okm0);  // loaded at the top
    __syncthreads();
    for (int it = 0; tile < g.ntiles; tile += gridDim.x, ++it) {
        uint16_t* cur = pl + (it & 1) * g.pbuf;
        uint16_t* nxt = pl + ((it + 1) & 1) * g.pbuf;
        const int64_t cimg = img;
        const int cp0 = p0, cq0 = q0;
        const bool more = tile + gridDim.x < g.ntiles;
        // next tile's loads (the current tile's again on the last pass, unused: no branch, so
        // nothing makes the compiler wait for them), consumed after the MFMAs and stores
        uint32_t pv[kElemsPerThread];
        origin(more ? tile + gridDim.x : tile, &img, &p0, &q0);
        const uint32_t okm =
            load_patch<CP, X32>(a, desc, (uint32_t)img * img_elems, p0 * a.sh - a.ph, q0 * a.sw - a.pw, pv);

        f32x16 acc[2][2];
        tile_mfma(cur, acc);
        // the next tile's patch goes to the other buffer now: its loads were issued before
        // the MFMAs, and waiting for them here does not also wait for this tile's stores
        if (more) write_patch(nxt, pv, okm);

        tile_epilogue(acc, cimg, cp0, cq0);
        __syncthreads();  // the next patch is complete; every wave is done with this one
    }
}

int pow2_at_least(int v) {
    int p = 1;
    while (p < v) p <<= 1;
    return p;
}

int round16(int v) { return (v + 15) & ~15; }

}  // namespace

bool conv_thin_plan(const ConvGemmArgs& a, ThinGeom* g) {
    if (a.apair || a.C > 8 || (!a.x_f32 && a.C % 8 == 0)) return false;
    ThinGeom t = {};
    t.CP = pow2_at_least(a.C);
    t.T = pow2_at_least(a.S * t.CP);
    if (t.T < 16) t.T = 16;
    t.logT = __builtin_ctz(t.T);
    t.RT = a.R * t.T;
    t.WPITCH = t.RT + 8;
    t.PH = (TP - 1) * a.sh + a.R;
    t.PW = (TQ - 1) * a.sw + (a.S > t.T / t.CP ? a.S : t.T / t.CP);
    t.tiles_p = (a.P + TP - 1) / TP;
    t.tiles_q = (a.Q + TQ - 1) / TQ;
    t.ntiles = (int64_t)a.N * t.tiles_p * t.tiles_q;
    const int64_t xelems = (int64_t)a.N * a.H * a.W * a.C;
    // large inputs (one million elements and up): zero-bordered copy + LDS-DMA patches, the
    // patch rows widened to whole 16-byte pieces; small ones (where a second launch would
    // cost more than it saves) load their patches element by element
    t.dma = xelems >= (1 << 20) ? 1 : 0;
    if (t.dma) {
        const int step = t.CP >= 8 ? 1 : 8 / t.CP;  // pixels per 16-byte piece
        t.PW = (t.PW + step - 1) / step * step;
        t.Hp = (t.tiles_p - 1) * TP * a.sh + t.PH;
        t.Wp = (t.tiles_q - 1) * TQ * a.sw + t.PW;
        if (t.Hp < a.H + a.ph) t.Hp = a.H + a.ph;
        if (t.Wp < a.W + a.pw) t.Wp = (a.W + a.pw + step - 1) / step * step;
        t.ppr = t.PW * t.CP / 8;
        t.npieces = t.PH * t.ppr;
        t.ni = (t.npieces + 255) / 256;
        t.ws_bytes = ((int64_t)a.N * t.Hp * t.Wp * t.CP * 2 + 255) / 256 * 256;
        if (t.ni > 8 || t.ws_bytes >= 0x7FFFFFF0ll) t.dma = 0;
    }
    if (!t.dma) {
        t.PW = (TQ - 1) * a.sw + (a.S > t.T / t.CP ? a.S : t.T / t.CP);
        t.ws_bytes = 0;
    }
    t.w_off = 0;
    t.p_off = round16(FB * t.WPITCH * 2);
    // bf16 elements per patch buffer: the patch (DMA: every piece the copies write)
    t.pbuf = t.dma ? t.ni * 256 * 8 : round16(t.PH * t.PW * t.CP * 2) / 2;
    t.s_off = t.p_off + 2 * t.pbuf * 2;
    t.lds_bytes = t.s_off + 4 * 32 * SPITCH * 4;
    const int nb = (a.R * a.S * a.C + 63) / 64;  // code blocks staged in the epilogue area
    t.rowlen = t.PW * a.C;
    t.nelem = t.PH * t.rowlen;
    t.ept = (t.nelem + 255) / 256;
    if (t.ntiles >= 0x7FFFFFFFll) return false;
    t.div_pqt = make_fastdiv((uint32_t)(t.tiles_p * t.tiles_q));
    t.div_tq = make_fastdiv((uint32_t)t.tiles_q);
    t.div_rowlen = make_fastdiv((uint32_t)t.rowlen);
    t.div_c = make_fastdiv((uint32_t)a.C);
    if (t.lds_bytes > 96 * 1024 || a.R > 64 || t.T > 128 || nb * 1024 > 4 * 32 * SPITCH * 4 ||
        (!t.dma && t.ept > kElemsPerThread) || t.PH * t.PW * t.CP >= 0xFFFF || t.PH > 63 || t.PW > 1023 ||
        xelems >= 0x7FFFFFFF)
        return false;
    *g = t;
    return true;
}

hipError_t launch_conv_thin(const ConvGemmArgs& a, const ThinGeom& g, hipStream_t stream) {
    const bool x32 = a.x_f32 != 0;
    const int tt = g.T / 16;
    const void* fn = nullptr;
#define TBN_THIN_PICK(cp, x, t, d) \
    if (g.CP == cp && x32 == x && tt == t && (g.dma != 0) == d) fn = reinterpret_cast<const void*>(&conv_thin_kernel<cp, x, t, d>);
#define TBN_THIN_PICK_T(cp, x, d) TBN_THIN_PICK(cp, x, 1, d) TBN_THIN_PICK(cp, x, 2, d) TBN_THIN_PICK(cp, x, 4, d) TBN_THIN_PICK(cp, x, 8, d)
    TBN_THIN_PICK_T(1, true, false) TBN_THIN_PICK_T(2, true, false) TBN_THIN_PICK_T(4, true, false) TBN_THIN_PICK_T(8, true, false)
    TBN_THIN_PICK_T(1, false, false) TBN_THIN_PICK_T(2, false, false) TBN_THIN_PICK_T(4, false, false) TBN_THIN_PICK_T(8, false, false)
#undef TBN_THIN_PICK_T
#undef TBN_THIN_PICK
    if (g.dma) {
        // the DMA kernel reads the bf16 zero-bordered copy whatever the input dtype
#define TBN_THIN_PICK_D(cp, t) if (g.CP == cp && tt == t) fn = reinterpret_cast<const void*>(&conv_thin_kernel<cp, false, t, true>);
        TBN_THIN_PICK_D(1, 1) TBN_THIN_PICK_D(1, 2) TBN_THIN_PICK_D(1, 4) TBN_THIN_PICK_D(1, 8)
        TBN_THIN_PICK_D(2, 1) TBN_THIN_PICK_D(2, 2) TBN_THIN_PICK_D(2, 4) TBN_THIN_PICK_D(2, 8)
        TBN_THIN_PICK_D(4, 1) TBN_THIN_PICK_D(4, 2) TBN_THIN_PICK_D(4, 4) TBN_THIN_PICK_D(4, 8)
        TBN_THIN_PICK_D(8, 1) TBN_THIN_PICK_D(8, 2) TBN_THIN_PICK_D(8, 4) TBN_THIN_PICK_D(8, 8)
#undef TBN_THIN_PICK_D
        if (!a.partial) return hipErrorInvalidValue;
        const int64_t pix = (int64_t)a.N * g.Hp * g.Wp;
        const dim3 pgrid((unsigned)((pix + 255) / 256));
        uint16_t* xp = reinterpret_cast<uint16_t*>(a.partial);
#define TBN_PAD(cp, x) hipLaunchKernelGGL((thin_pad_kernel<cp, x>), pgrid, dim3(256), 0, stream, a, g, xp)
        switch (g.CP * 2 + (x32 ? 1 : 0)) {
            case 2: TBN_PAD(1, false); break;
            case 3: TBN_PAD(1, true); break;
            case 4: TBN_PAD(2, false); break;
            case 5: TBN_PAD(2, true); break;
            case 8: TBN_PAD(4, false); break;
            case 9: TBN_PAD(4, true); break;
            case 16: TBN_PAD(8, false); break;
            default: TBN_PAD(8, true); break;
        }
#undef TBN_PAD
        const hipError_t pe = hipGetLastError();
        if (pe != hipSuccess) return pe;
    }
    if (!fn) return hipErrorInvalidValue;
    if (g.lds_bytes > 65536 &&
        hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, g.lds_bytes) != hipSuccess)
        return hipErrorInvalidConfiguration;
    // persistent blocks: as many as can be resident at once (one round), each walking tiles
    int per_cu = 0, dev = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, 256, g.lds_bytes) != hipSuccess || per_cu < 1)
        per_cu = 1;
    if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) !=
                                                 hipSuccess || cus < 1)
        cus = 256;
    const int kb = (a.Kf + FB - 1) / FB;
    int64_t cap = (int64_t)per_cu * cus / kb;
    if (cap < 1) cap = 1;
    const dim3 grid((unsigned)(g.ntiles < cap ? g.ntiles : cap), (unsigned)kb);
    ConvGemmArgs ka = a;
    ThinGeom kg = g;
    void* args[] = {&ka, &kg};
    return hipLaunchKernel(fn, grid, dim3(256), args, (size_t)g.lds_bytes, stream);
}

}  // namespace tbn
