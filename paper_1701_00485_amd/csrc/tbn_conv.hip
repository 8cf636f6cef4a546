// tbn_conv.hip -- implicit-GEMM convolution on bf16 MFMA with the two-bit filters decoded
// in registers.  One kernel template serves
//   * the forward pass (Sec. 2 Eq. 1; Algorithm 1 forward step): rows = output pixels
//     (n,p,q), columns = filters k, reduction = filter elements (r,s,c); every code is
//     decoded to an exact bf16 +-1/+-2 and alpha_k is applied to the fp32 sum; and
//   * the backward-data pass (Sec. 3, backward through the approximate filters): the
//     same GEMM over dy with the transposed, spatially flipped filter, whose codes are
//     decoded straight into bf16(alpha_k) * W~ (sign flip / exponent + 1 of the scale).
//
// Work split (256 threads = 4 waves of 64, CDNA4):
//   * the block owns a BM x BN output tile; each wave a WM x WN sub-tile made of 32x32
//     v_mfma_f32_32x32x16_bf16 tiles with fp32 accumulators;
//   * the reduction advances 64 elements per stage, which is exactly one 1 KiB block of
//     packed codes per 64 filters;
//   * the activation tile (BM rows x 64 elements, bf16) is gathered from NHWC memory
//     (zero padding by predication) into LDS, double buffered, rows padded by 8 bf16 so
//     the 16-byte MFMA operand reads do not conflict;
//   * the filter operand never touches LDS: lane l of a wave loads the four words of
//     filter (l % 32) of its 32-column group (one coalesced 16-byte load per lane, 512
//     bytes per wave) and decodes at each 16-element MFMA step the 8 elements the MFMA
//     B layout gives it (elements 8*(l/32)..+7 of the step) with 2 integer ops per pair.
#include <cstdlib>

#include "tbn_device.h"
#include "tbn_kernels.h"

namespace tbn {

namespace {

constexpr int BK = 64;       // reduction elements per stage
constexpr int LDA = BK + 8;  // LDS row pitch (bf16 elements)

enum { A_VEC8 = 0, A_SCALAR = 1 };

template <int BM, int BN, int WM, int WN, int AM, bool BWD>
__global__ __launch_bounds__(256) void conv_gemm_kernel(const ConvGemmArgs a) {
    constexpr int WAVES_N = BN / WN;
    static_assert((BM / WM) * (BN / WN) == 4, "four waves per block");
    constexpr int TM = WM / 32, TN = WN / 32;

    __shared__ __attribute__((aligned(16))) uint16_t As[2][BM * LDA];
    // Row table of the scalar gather: image offset and top-left input coordinate.
    __shared__ int64_t row_img[AM == A_SCALAR ? BM : 1];
    __shared__ int32_t row_h[AM == A_SCALAR ? BM : 1];
    __shared__ int32_t row_w[AM == A_SCALAR ? BM : 1];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / WAVES_N;
    const int wn = wave % WAVES_N;
    const int half = lane >> 5;  // which 8 of a 16-element MFMA step this lane holds
    const int l32 = lane & 31;

    const int64_t PQ = (int64_t)a.P * a.Q;
    const int64_t M = (int64_t)a.N * PQ;
    const int C = a.C;
    const int n = a.R * a.S * C;
    const int nchunks = (n + BK - 1) / BK;
    const int KB = (a.Kf + 63) / 64;
    const int tilesN = (a.Kf + BN - 1) / BN;
    // XCD-aware order: each XCD runs a contiguous range of tiles (column tiles of one row
    // tile first), so the activation rows and halos a tile re-reads stay in one L2.
    const int64_t tile = xcd_remap(blockIdx.x, gridDim.x);
    const int64_t tm = tile / tilesN;
    const int tn = (int)(tile % tilesN);
    const int64_t m0 = tm * BM;
    const int n0 = tn * BN;
    const int64_t HWC = (int64_t)a.H * a.W * C;

    // ---------------- activation gather state ----------------
    constexpr int AR = (AM == A_VEC8) ? BM / 32 : BM / 4;  // rows per thread
    const int seg = tid & 7;        // A_VEC8: 16-byte segment of the 64-element row
    const int vrow = tid >> 3;      // A_VEC8: first row
    const int sel = tid & 63;       // A_SCALAR: element of the chunk
    const int srow = tid >> 6;      // A_SCALAR: first row
    int32_t rh[AM == A_VEC8 ? AR : 1], rw[AM == A_VEC8 ? AR : 1];
    int64_t rimg[AM == A_VEC8 ? AR : 1];
    if constexpr (AM == A_VEC8) {
#pragma unroll
        for (int j = 0; j < AR; ++j) {
            const int64_t m = m0 + vrow + 32 * j;
            if (m < M) {
                const int64_t img = m / PQ;
                const int pq = (int)(m - img * PQ);
                const int p = pq / a.Q, q = pq - (pq / a.Q) * a.Q;
                rimg[j] = img * HWC;
                rh[j] = p * a.sh - a.ph;
                rw[j] = q * a.sw - a.pw;
            } else {
                rimg[j] = 0;
                rh[j] = -0x40000000;  // never inside the image
                rw[j] = -0x40000000;
            }
        }
    } else {
        for (int r = tid; r < BM; r += 256) {
            const int64_t m = m0 + r;
            if (m < M) {
                const int64_t img = m / PQ;
                const int pq = (int)(m - img * PQ);
                const int p = pq / a.Q, q = pq - (pq / a.Q) * a.Q;
                row_img[r] = img * HWC;
                row_h[r] = p * a.sh - a.ph;
                row_w[r] = q * a.sw - a.pw;
            } else {
                row_img[r] = 0;
                row_h[r] = -0x40000000;
                row_w[r] = -0x40000000;
            }
        }
        __syncthreads();
    }
    // (r, s, c) of this thread's first element in the current chunk (A_VEC8)
    int er = 0, es = 0, ec = 0;
    if constexpr (AM == A_VEC8) {
        const int e0 = seg * 8;
        const int rs = e0 / C;
        ec = e0 - rs * C;
        er = rs / a.S;
        es = rs - er * a.S;
    }

    u32x4 areg[AM == A_VEC8 ? AR : 1];
    uint16_t sreg[AM == A_SCALAR ? AR : 1];

    auto load_a = [&](int chunk) {
        if constexpr (AM == A_VEC8) {
            const uint16_t* x = reinterpret_cast<const uint16_t*>(a.x);
#pragma unroll
            for (int j = 0; j < AR; ++j) {
                u32x4 v = {0u, 0u, 0u, 0u};
                const int h = rh[j] + er, w = rw[j] + es;
                if (er < a.R && (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W)
                    v = *reinterpret_cast<const u32x4*>(x + rimg[j] + ((int64_t)h * a.W + w) * C + ec);
                areg[j] = v;
            }
        } else {
            const int e = chunk * BK + sel;
            int r = 0, s = 0, c = 0;
            const bool ok = e < n;
            if (ok) {
                const int rs = e / C;
                c = e - rs * C;
                r = rs / a.S;
                s = rs - r * a.S;
            }
#pragma unroll 4
            for (int j = 0; j < AR; ++j) {
                const int row = srow + 4 * j;
                uint16_t v = 0;
                const int h = row_h[row] + r, w = row_w[row] + s;
                if (ok && (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W) {
                    const int64_t off = row_img[row] + ((int64_t)h * a.W + w) * C + c;
                    if (a.x_f32)
                        v = (uint16_t)f32_to_bf16_bits(reinterpret_cast<const float*>(a.x)[off]);
                    else
                        v = reinterpret_cast<const uint16_t*>(a.x)[off];
                }
                sreg[j] = v;
            }
        }
    };
    auto advance_a = [&]() {
        if constexpr (AM == A_VEC8) {
            ec += BK;
            while (ec >= C) {
                ec -= C;
                if (++es == a.S) {
                    es = 0;
                    ++er;
                }
            }
        }
    };
    auto store_a = [&](int buf) {
        if constexpr (AM == A_VEC8) {
#pragma unroll
            for (int j = 0; j < AR; ++j)
                *reinterpret_cast<u32x4*>(&As[buf][(vrow + 32 * j) * LDA + seg * 8]) = areg[j];
        } else {
#pragma unroll
            for (int j = 0; j < AR; ++j) As[buf][(srow + 4 * j) * LDA + sel] = sreg[j];
        }
    };

    // ---------------- filter operand state ----------------
    u32x4 braw[TN];
    u32x4 bnext[TN];
    u32x4 base[4];
    u32x4 base_next[4];
    auto load_b = [&](int chunk, u32x4* dst, u32x4* bdst) {
#pragma unroll
        for (int t = 0; t < TN; ++t) {
            const int f = n0 + wn * WN + 32 * t + l32;
            const int fb = f >> 6;
            u32x4 v = {0u, 0u, 0u, 0u};
            if (fb < KB)
                v = *reinterpret_cast<const u32x4*>(a.codes + (((int64_t)fb * nchunks + chunk) * 64 + (f & 63)) * 4);
            dst[t] = v;
        }
        if constexpr (BWD) {
#pragma unroll
            for (int u = 0; u < 4; ++u)
                bdst[u] = *reinterpret_cast<const u32x4*>(a.apair + (int64_t)chunk * 32 + 8 * u + 4 * half);
        }
    };
    if constexpr (!BWD) {
#pragma unroll
        for (int u = 0; u < 4; ++u) base[u] = u32x4{0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u};
    }

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int t = 0; t < TN; ++t)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][t][v] = 0.0f;

    // ---------------- main loop ----------------
    load_a(0);
    load_b(0, braw, base);
    store_a(0);
    __syncthreads();
    for (int chunk = 0; chunk < nchunks; ++chunk) {
        const int cur = chunk & 1;
        const bool more = chunk + 1 < nchunks;
        if (more) {
            advance_a();
            load_a(chunk + 1);
            load_b(chunk + 1, bnext, base_next);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            bf16x8 af[TM];
#pragma unroll
            for (int i = 0; i < TM; ++i)
                af[i] = *reinterpret_cast<const bf16x8*>(
                    &As[cur][(wm * WM + 32 * i + l32) * LDA + 16 * u + 8 * half]);
            bf16x8 bfr[TN];
#pragma unroll
            for (int t = 0; t < TN; ++t) {
                const uint32_t wd = braw[t][u] >> (4 * half);
                bfr[t] = as_bf16x8(decode8(wd, base[u]));
            }
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int t = 0; t < TN; ++t) acc[i][t] = mfma32(af[i], bfr[t], acc[i][t]);
        }
        if (more) {
            store_a(cur ^ 1);
#pragma unroll
            for (int t = 0; t < TN; ++t) braw[t] = bnext[t];
            if constexpr (BWD) {
#pragma unroll
                for (int u = 0; u < 4; ++u) base[u] = base_next[u];
            }
        }
        __syncthreads();
    }

    // ---------------- epilogue ----------------
    const int Kf = a.Kf;
#pragma unroll
    for (int t = 0; t < TN; ++t) {
        const int col = n0 + wn * WN + 32 * t + l32;
        if (col >= Kf) continue;
        float cs = a.colscale ? a.colscale[col] : 1.0f;
        if (a.scale) cs *= a.scale[col];
        const float bi = a.bias ? a.bias[col] : 0.0f;
#pragma unroll
        for (int i = 0; i < TM; ++i) {
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int64_t row = m0 + wm * WM + 32 * i + 8 * (v >> 2) + 4 * half + (v & 3);
                if (row >= M) continue;
                const int64_t o = row * Kf + col;
                float val = acc[i][t][v] * cs + bi;
                if (a.residual) {
                    val += a.y_f32 ? reinterpret_cast<const float*>(a.residual)[o]
                                   : bf16_bits_to_f32(reinterpret_cast<const uint16_t*>(a.residual)[o]);
                }
                if (a.relu) val = fmaxf(val, 0.0f);
                if (a.y_f32)
                    reinterpret_cast<float*>(a.y)[o] = val;
                else
                    reinterpret_cast<uint16_t*>(a.y)[o] = (uint16_t)f32_to_bf16_bits(val);
            }
        }
    }
}

template <int BM, int BN, int WM, int WN, int AM, bool BWD>
hipError_t launch_cfg(const ConvGemmArgs& a, hipStream_t stream) {
    const int64_t M = (int64_t)a.N * a.P * a.Q;
    const int64_t tiles = ((M + BM - 1) / BM) * ((a.Kf + BN - 1) / BN);
    if (tiles > 0x7FFFFFFF) return hipErrorInvalidValue;
    hipLaunchKernelGGL((conv_gemm_kernel<BM, BN, WM, WN, AM, BWD>), dim3((unsigned)tiles), dim3(256), 0,
                       stream, a);
    return hipGetLastError();
}


template <int AM, bool BWD>
hipError_t launch_mode(const ConvGemmArgs& a, int cfg, hipStream_t stream) {
    if (cfg == 1 || (cfg < 0 && a.Kf <= 64)) return launch_cfg<256, 64, 64, 64, AM, BWD>(a, stream);
    return launch_cfg<128, 128, 64, 64, AM, BWD>(a, stream);
}

// ---------------- backward-data operand preparation ----------------
// K may exceed the layer's Kreal filters (a gradient padded to a multiple of 8 channels):
// filters k >= Kreal read the zero padding bits of the last 64-filter block and get scale 0.
__global__ __launch_bounds__(256) void repack_bwd_kernel(const uint32_t* __restrict__ codes,
                                                         const float* __restrict__ alpha, int32_t K, int32_t Kreal,
                                                         int32_t R, int32_t S, int32_t C,
                                                         uint32_t* __restrict__ codes_t,
                                                         uint32_t* __restrict__ apair) {
    // every count below is < 2^31 (R*S*C and R*S*K < 2^30, checked by the host)
    const uint32_t n = (uint32_t)(R * S * C);     // elements of a forward filter
    const uint32_t nt = (uint32_t)(R * S * K);    // elements of a transposed filter
    const uint32_t nb = (n + 63) / 64;
    const uint32_t nbt = (nt + 63) / 64;
    const uint32_t cb = (uint32_t)(C + 63) / 64;
    const int64_t words = (int64_t)cb * nbt * 256;
    const int64_t pairs = (int64_t)nbt * 32;
    const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (gid < words) {
        const uint32_t g32 = (uint32_t)gid;
        const uint32_t wsub = g32 & 3;
        const uint32_t cc = (g32 >> 2) & 63;
        const uint32_t eb = (g32 >> 8) % nbt;
        const uint32_t cblk = (g32 >> 8) / nbt;
        const uint32_t c = cblk * 64 + cc;
        uint32_t word = 0;
        uint32_t et = eb * 64 + wsub * 16;  // first (r', s', k) of the flipped filter in this word
        if (c < (uint32_t)C && et < nt) {
            // walk k, carrying into s' and r' (one division per word, none per element)
            uint32_t k = et % (uint32_t)K, rs = et / (uint32_t)K;
            uint32_t rp = rs / (uint32_t)S, sp = rs - rp * (uint32_t)S;
            for (int e = 0; e < 16 && et < nt; ++e, ++et) {
                const uint32_t i = ((R - 1 - rp) * S + (S - 1 - sp)) * C + c;  // element of forward filter k
                const uint32_t src = codes[(((k >> 6) * nb + (i >> 6)) * 64 + (k & 63)) * 4 + ((i & 63) >> 4)];
                const int ei = (int)(i & 15), hi = ei & 1, j = ei >> 1;
                const uint32_t mag = (src >> (16 * hi + j)) & 1u;
                const uint32_t neg = (src >> (16 * hi + 8 + j)) & 1u;
                const int eh = e & 1, ej = e >> 1;
                word |= (mag << (16 * eh + ej)) | (neg << (16 * eh + 8 + ej));
                if (++k == (uint32_t)K) {
                    k = 0;
                    if (++sp == (uint32_t)S) {
                        sp = 0;
                        ++rp;
                    }
                }
            }
        }
        codes_t[gid] = word;
    }
    if (gid < pairs) {
        uint32_t v = 0;
        for (int h = 0; h < 2; ++h) {
            const uint32_t et = 2 * (uint32_t)gid + h;
            if (et < nt) {
                const uint32_t kk = et % (uint32_t)K;
                uint32_t b = kk < (uint32_t)Kreal ? f32_to_bf16_bits(alpha[kk]) : 0u;
                if ((b & 0x7F80u) == 0) b = 0;  // a denormal scale is flushed: exponent + 1 would not double it
                v |= b << (16 * h);
            }
        }
        apair[gid] = v;
    }
}

}  // namespace

// Tile-shape and split overrides for tuning and for the tests that cover every shape (the
// knobs of tbn_tuning.h; -1 = the built-in choice).
int conv_tile_override() { return knob(KNOB_CONV_TILE); }

int conv_splits_override() { return knob(KNOB_CONV_SPLITS); }

// Which kernel runs a forward / backward-data GEMM: the weight-streaming kernel for a
// fully-connected layer of at most 16 rows, the LDS-DMA implicit GEMM for C % 8 == 0, the
// direct kernel for small few-channel layers, the thin-input kernel for other few-channel
// ones, else the general one.  cfg (the tile knob) forces a family: 0-1 general, 10-19 and
// 21-25 LDS-DMA tile shapes, 20 thin, 30 weight streaming, 40 direct.
enum ConvPath { PATH_FC, PATH_DMA, PATH_DIRECT, PATH_THIN, PATH_GENERIC };

static ConvPath choose_path(const ConvGemmArgs& a, int cfg, FcStreamPlan* fp, ThinGeom* tg) {
    if ((cfg < 0 || cfg == 30) && fc_stream_plan(a, fp)) return PATH_FC;
    if (conv_dma_eligible(a) && (cfg < 0 || (cfg >= 10 && cfg < 20) || (cfg >= 21 && cfg <= 25))) return PATH_DMA;
    if ((cfg < 0 || cfg == 40) && conv_direct_eligible(a)) return PATH_DIRECT;
    if ((cfg < 0 || cfg == 20) && conv_thin_plan(a, tg)) return PATH_THIN;
    return PATH_GENERIC;
}

size_t conv_gemm_partial_bytes(const ConvGemmArgs& a) {
    const int cfg = conv_tile_override();
    FcStreamPlan fp;
    ThinGeom tg;
    switch (choose_path(a, cfg, &fp, &tg)) {
        case PATH_DMA: return plan_conv_dma(a, cfg).partial_bytes;
        case PATH_THIN: return tg.dma ? (size_t)tg.ws_bytes : 0;
        default: return 0;
    }
}

hipError_t launch_conv_gemm(const ConvGemmArgs& args, hipStream_t stream) {
    ConvGemmArgs a = args;
    a.div_q = make_fastdiv((uint32_t)a.Q);
    a.div_pq = make_fastdiv((uint32_t)a.P * (uint32_t)a.Q);
    a.splits = 1;
    a.chunks_per_split = 1 << 30;
    const int cfg = conv_tile_override();
    FcStreamPlan fp;
    ThinGeom tg;
    switch (choose_path(a, cfg, &fp, &tg)) {
        case PATH_FC: return launch_fc_stream(a, fp, stream);
        case PATH_DMA: return launch_conv_dma(a, plan_conv_dma(a, cfg), stream);
        case PATH_DIRECT: return launch_conv_direct(a, stream);
        case PATH_THIN: return launch_conv_thin(a, tg, stream);
        default: break;
    }
    const bool vec = (a.C % 8 == 0) && !a.x_f32;
    if (a.apair) return vec ? launch_mode<A_VEC8, true>(a, cfg, stream) : launch_mode<A_SCALAR, true>(a, cfg, stream);
    return vec ? launch_mode<A_VEC8, false>(a, cfg, stream) : launch_mode<A_SCALAR, false>(a, cfg, stream);
}

hipError_t launch_repack_bwd(const uint32_t* codes, const float* alpha, int32_t K, int32_t Kreal, int32_t R,
                             int32_t S, int32_t C, uint32_t* codes_t, uint32_t* apair, hipStream_t stream) {
    const int64_t nt = (int64_t)R * S * K;
    const int64_t nbt = (nt + 63) / 64;
    const int64_t words = (int64_t)((C + 63) / 64) * nbt * 256;
    const int64_t total = words > nbt * 32 ? words : nbt * 32;
    hipLaunchKernelGGL(repack_bwd_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, stream, codes,
                       alpha, K, Kreal, R, S, C, codes_t, apair);
    return hipGetLastError();
}

}  // namespace tbn
