// tbn_wgrad_dma.hip -- gradient with respect to the approximate filter (Algorithm 1,
// backward step; Sec. 3 applies it unchanged to the real weights):
//     dW[k][j] = sum_m dy[m][k] * x_col[m][j],   m = (n,p,q) output pixel, j = (r,s,c),
// for bf16 activations with C % 8 == 0 and K % 8 == 0.
//
// Both operands arrive with the reduction index (the pixel) outermost, while the MFMA
// wants 8 consecutive reduction elements per lane.  Instead of transposing in registers,
// the kernels copy the raw tiles into LDS with LDS-DMA buffer loads and form the MFMA
// operands with the gfx950 transposing LDS read (ds_read_b64_tr_b16: a 16-lane group
// turns a 16 x 4 block of 16-bit values into 4 consecutive rows per lane), so the main
// loop spends no vector ALU work on data movement:
//   * a block of 8 waves owns a 256 (k) x 256 (j) output tile; each wave 128 x 64 made of
//     32x32 v_mfma_f32_32x32x16_bf16 tiles with fp32 accumulators;
//   * a stage is 64 pixels, two stages in LDS: the DMAs of stage c+1 overlap the MFMAs of
//     stage c, and the operands of each 16-pixel step are read during the previous one;
//   * the pixel range is split over the grid (split-K): each split writes fp32 partials
//     that a second kernel adds in a fixed order (deterministic result).
// Two stage layouts:
//   * pixel-major (wide layers): each pixel's 256 dy channels / 256 x columns form one
//     row of the stage, padded to 576 bytes; one DMA instruction copies one pixel's 512
//     contiguous bytes, so the requests cover whole cache lines;
//   * segment-major (K < 128): for every 8-channel segment the 64 pixels' 16-byte pieces
//     are contiguous (one DMA instruction, lane = pixel), segments 1088 bytes apart; with
//     few valid dy channels this issues fewer copies.
#include <cstdlib>

#include "tbn_device.h"
#include "tbn_dma.h"
#include "tbn_kernels.h"

namespace tbn {

namespace {

constexpr int SEGS = 32;             // 8-channel segments of the dy tile (256 channels)
constexpr int TILE_K = 256;

// Stage geometry: PIXS pixels per stage; each 8-channel segment holds the PIXS pixels'
// 16-byte pieces contiguously, segments padded by 64 bytes (bank spread of the
// transposing reads of neighbouring segments).  A stage holds the 32 dy segments, then
// the 8 WN x segments (TILE_J = 64 WN columns).
template <int PIXS, int WN>
struct WgStage {
    static constexpr int SEG_PITCH = PIXS * 16 + 64;
    static constexpr int OP_BYTES = SEGS * SEG_PITCH;          // dy tile
    static constexpr int BYTES = (SEGS + 8 * WN) * SEG_PITCH;  // dy tile then x tile
};

struct WgradDmaArgs {
    WgradArgs a;
    FastDiv div_q, div_pq;
};

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;

__device__ __forceinline__ v4i16 read_tr(uint32_t addr) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(uintptr_t)addr);
}

// 8 consecutive pixels of one channel as an MFMA operand (two transposing reads).
__device__ __forceinline__ bf16x8 operand(uint32_t addr) {
    const v4i16 lo = read_tr(addr);
    const v4i16 hi = read_tr(addr + 64);  // pixels + 4
    typedef short v8i16 __attribute__((ext_vector_type(8)));
    const v8i16 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    return __builtin_bit_cast(bf16x8, v);
}

// Segment-major variant: 64-pixel stages, two-deep LDS ring, 2 x 4 waves (wave tile
// 128 x 64, block tile 256 x 256).
__global__ __launch_bounds__(512, 1) void wgrad_seg_kernel(const WgradDmaArgs ka) {
    constexpr int PIXS = 64, STAGES = 2, WN = 4;
    const WgradArgs& a = ka.a;
    constexpr int TM = 4, TN = 2;  // wave tile 128 x 64
    constexpr int TILE_J = 64 * WN;
    constexpr int DYQ = SEGS / (2 * WN);  // dy segments each wave copies
    using L = WgStage<PIXS, WN>;
    constexpr int SEG_PITCH = L::SEG_PITCH;
    constexpr int OP_BYTES = L::OP_BYTES;

    __shared__ __attribute__((aligned(1024))) uint8_t smem[STAGES * L::BYTES];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / WN;  // 0..1
    const int wn = wave % WN;

    const int K = a.K, C = a.C;
    const int J = a.R * a.S * C;
    const uint32_t PQ = (uint32_t)a.P * a.Q;
    const int64_t M = (int64_t)a.N * PQ;
    const int64_t nchunks = (M + PIXS - 1) / PIXS;
    const int tilesJ = (J + TILE_J - 1) / TILE_J;
    const int tiles = tilesJ * ((K + TILE_K - 1) / TILE_K);
    const int t_ = (int)xcd_remap(blockIdx.x, gridDim.x);
    const int split = t_ / tiles;
    const int k0 = ((t_ % tiles) / tilesJ) * TILE_K;
    const int j0 = ((t_ % tiles) % tilesJ) * TILE_J;
    const int64_t c_begin = (int64_t)split * a.chunks_per_split;  // 64-pixel chunks
    const int64_t c_end = min(c_begin + (int64_t)a.chunks_per_split, nchunks);

    const v4i rs_dy = make_rsrc(a.dy, (uint32_t)(M * K * 2));
    const v4i rs_x = make_rsrc(a.x, (uint32_t)((int64_t)a.N * a.H * a.W * C * 2));
    const uint32_t smem_base = lds_addr(smem);

    // segments this wave copies: DYQ of dy (channels k0 + 8 sg) and 4 of x (columns j0 + 8 sg)
    int xr[4], xs[4], xc[4];
    bool dy_ok[DYQ], x_ok[4];
#pragma unroll
    for (int q = 0; q < DYQ; ++q) dy_ok[q] = k0 + 8 * (DYQ * wave + q) < K;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int sg = 4 * wave + q;
        const int j = j0 + 8 * sg;
        x_ok[q] = j < J;
        const int rs = x_ok[q] ? j / C : 0;
        xc[q] = x_ok[q] ? j - rs * C : 0;
        xr[q] = rs / a.S;
        xs[q] = rs - xr[q] * a.S;
    }
    const int64_t HWC = (int64_t)a.H * a.W * C;

    const int px = lane;  // lane = pixel of the stage for every DMA
    auto issue = [&](int64_t chunk) {
        const uint32_t st = smem_base + (uint32_t)((chunk % STAGES) * L::BYTES);
        const int64_t m = chunk * PIXS + px;
        const bool mok = m < M;
        const uint32_t mm = mok ? (uint32_t)m : 0u;
        const uint32_t img = fdiv(mm, ka.div_pq);
        const uint32_t pq = mm - img * PQ;
        const uint32_t p = fdiv(pq, ka.div_q);
        const uint32_t q_ = pq - p * (uint32_t)a.Q;
        const int h0 = (int)p * a.sh - a.ph, w0 = (int)q_ * a.sw - a.pw;
        const uint32_t dy_row = mm * (uint32_t)K * 2u;
        const uint32_t x_img = (uint32_t)(img * HWC);
#pragma unroll
        for (int q = 0; q < DYQ; ++q) {
            const int sg = DYQ * wave + q;
            const uint32_t off = (mok && dy_ok[q]) ? dy_row + (uint32_t)(k0 + 8 * sg) * 2u : 0x80000000u;
            dma_b128(rs_dy, st + (uint32_t)(sg * SEG_PITCH), off);
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int sg = 4 * wave + q;
            const int h = h0 + xr[q], w = w0 + xs[q];
            const bool ok = mok && x_ok[q] && (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W;
            const uint32_t off = ok ? (x_img + (uint32_t)((h * a.W + w) * C + xc[q])) * 2u : 0x80000000u;
            dma_b128(rs_x, st + (uint32_t)(OP_BYTES + sg * SEG_PITCH), off);
        }
    };
    constexpr int kDmas = DYQ + 4;  // DMA instructions per wave per stage

    // transposing-read addressing: lane (group g = lane / 16, i = lane % 16) reads the
    // 8 bytes at channel 16 (g % 2) + 4 (i % 4) of pixel 8 (g / 2) + i / 4 (+ 4 for the
    // second read) relative to the 32-channel tile and the 16-pixel step
    const int g = lane >> 4, i16 = lane & 15;
    const int chl = 16 * (g & 1) + 4 * (i16 & 3);
    const uint32_t lane_off = (uint32_t)((chl >> 3) * SEG_PITCH + (chl & 7) * 2 + (8 * (g >> 1) + (i16 >> 2)) * 16);
    const uint32_t a_base = (uint32_t)(((wm * 128) >> 3) * SEG_PITCH) + lane_off;            // dy rows
    const uint32_t b_base = (uint32_t)(OP_BYTES + ((wn * 64) >> 3) * SEG_PITCH) + lane_off;   // x columns

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int t = 0; t < TN; ++t)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][t][v] = 0.0f;

#pragma unroll
    for (int c = 0; c < STAGES - 1; ++c)
        if (c_begin + c < c_end) issue(c_begin + c);
    for (int64_t chunk = c_begin; chunk < c_end; ++chunk) {
        // this wave's DMAs of stage `chunk` landed (later stages may still be in flight)
        const int later = (int)min(c_end - 1 - chunk, (int64_t)(STAGES - 2));
        wait_vmcnt(later * kDmas);
        __syncthreads();  // ... and every other wave's; all reads of stage chunk-1 are done
        if (chunk + STAGES - 1 < c_end) issue(chunk + STAGES - 1);  // into stage chunk-1's buffer
        const uint32_t st = smem_base + (uint32_t)((chunk % STAGES) * L::BYTES);
        // operands of 16-pixel step u + 1 are read while the MFMAs of step u run
        bf16x8 af[2][TM], bf[2][TN];
        auto load = [&](int u, int b) {
#pragma unroll
            for (int i = 0; i < TM; ++i) af[b][i] = operand(st + a_base + (uint32_t)(4 * i * SEG_PITCH + u * 256));
#pragma unroll
            for (int t = 0; t < TN; ++t) bf[b][t] = operand(st + b_base + (uint32_t)(4 * t * SEG_PITCH + u * 256));
        };
        load(0, 0);
#pragma unroll
        for (int u = 0; u < PIXS / 16; ++u) {
            if (u + 1 < PIXS / 16) load(u + 1, (u + 1) & 1);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int t = 0; t < TN; ++t) acc[i][t] = mfma32(af[u & 1][i], bf[u & 1][t], acc[i][t]);
        }
    }

    float* out = a.out + (int64_t)split * K * J;
    const int l32 = lane & 31, half = lane >> 5;
#pragma unroll
    for (int t = 0; t < TN; ++t) {
        const int col = j0 + wn * 32 * TN + 32 * t + l32;
        if (col >= J) continue;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int row = k0 + wm * 128 + 32 * i + 8 * (v >> 2) + 4 * half + (v & 3);
                if (row < K) {
                    float* o = out + (int64_t)row * J + col;
                    *o = a.accumulate ? *o + acc[i][t][v] : acc[i][t][v];
                }
            }
    }
}

// Pixel-major variant: a stage holds PIXR pixels of the dy tile (256 channels, 512 bytes)
// then the same pixels of the x tile (256 columns), each pixel row padded to 576 bytes
// (with that pitch the transposing reads below use every LDS bank exactly twice).  One
// DMA instruction copies one pixel's 512 contiguous bytes (lanes 0..31, 16 bytes each),
// so every request covers whole 128-byte lines; the per-pixel address arithmetic is
// wave-uniform and each lane's channel / tap offset is fixed for the whole kernel.
constexpr int PPITCH = 576;

// PIXR pixels per stage, STAGES-deep ring.
template <int PIXR, int STAGES>
__global__ __launch_bounds__(512, 1) void wgrad_rows_kernel(const WgradDmaArgs ka) {
    const WgradArgs& a = ka.a;
    constexpr int WNW = 4;          // waves along j (2 x 4 waves)
    constexpr int TM = 4, TN = 2;   // wave tile 128 x 64 of the 256 x 256 block tile
    constexpr int PPW = PIXR / 8;   // pixels each wave copies per stage
    constexpr int PR_OP = PIXR * PPITCH;  // one operand tile of a stage
    constexpr int PR_STAGE = 2 * PR_OP;

    __shared__ __attribute__((aligned(1024))) uint8_t smem[STAGES * PR_STAGE];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / WNW;
    const int wn = wave % WNW;

    const int K = a.K, C = a.C;
    const int J = a.R * a.S * C;
    const uint32_t PQ = (uint32_t)a.P * a.Q;
    const int64_t M = (int64_t)a.N * PQ;
    const int64_t nchunks = (M + PIXR - 1) / PIXR;
    const int tilesJ = (J + 255) / 256;
    const int tiles = tilesJ * ((K + 255) / 256);
    const int t_ = (int)xcd_remap(blockIdx.x, gridDim.x);
    const int split = t_ / tiles;
    const int k0 = ((t_ % tiles) / tilesJ) * 256;
    const int j0 = ((t_ % tiles) % tilesJ) * 256;
    // the split ranges are given in 64-pixel chunks
    const int64_t c_begin = (int64_t)split * a.chunks_per_split * (64 / PIXR);
    const int64_t c_end = min(c_begin + (int64_t)a.chunks_per_split * (64 / PIXR), nchunks);

    const v4i rs_dy = make_rsrc(a.dy, (uint32_t)(M * K * 2));
    const v4i rs_x = make_rsrc(a.x, (uint32_t)((int64_t)a.N * a.H * a.W * C * 2));
    const uint32_t smem_base = lds_addr(smem);

    // this lane's 8-channel segment of the dy row and of the x column tile
    const int seg = lane & 31;
    const bool dy_ok = k0 + 8 * seg < K;
    const uint32_t dy_col = (uint32_t)(k0 + 8 * seg) * 2u;
    const int jx = j0 + 8 * seg;
    const bool x_ok = jx < J;
    const int rsx = x_ok ? jx / C : 0;
    const int xc = x_ok ? jx - rsx * C : 0;
    const int xr = rsx / a.S, xs = rsx - (rsx / a.S) * a.S;
    const int64_t HWC = (int64_t)a.H * a.W * C;

    auto issue = [&](int64_t chunk) {
        const uint32_t st = smem_base + (uint32_t)((chunk % STAGES) * PR_STAGE);
        if (lane < 32) {
#pragma unroll
            for (int pp = 0; pp < PPW; ++pp) {
                const int pl = PPW * wave + pp;  // pixel of the stage (wave-uniform)
                const int64_t m = chunk * PIXR + pl;
                const bool mok = m < M;
                const uint32_t mm = mok ? (uint32_t)m : 0u;
                const uint32_t img = fdiv(mm, ka.div_pq);
                const uint32_t pq = mm - img * PQ;
                const uint32_t p = fdiv(pq, ka.div_q);
                const uint32_t q_ = pq - p * (uint32_t)a.Q;
                const int h = (int)p * a.sh - a.ph + xr, w = (int)q_ * a.sw - a.pw + xs;
                const uint32_t offd = (mok && dy_ok) ? mm * (uint32_t)K * 2u + dy_col : 0x80000000u;
                dma_b128(rs_dy, st + (uint32_t)(pl * PPITCH), offd);
                const bool ok = mok && x_ok && (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W;
                const uint32_t offx = ok ? ((uint32_t)(img * HWC) + (uint32_t)((h * a.W + w) * C + xc)) * 2u : 0x80000000u;
                dma_b128(rs_x, st + (uint32_t)(PR_OP + pl * PPITCH), offx);
            }
        }
    };
    constexpr int kDmas = 2 * PPW;

    // transposing reads: lane (g = lane / 16, i = lane % 16) reads the 8 bytes of channels
    // 16 (g % 2) + 4 (i % 4) .. + 3 of pixel 8 (g / 2) + i / 4 (+ 4 for the second read)
    const int g = lane >> 4, i16 = lane & 15;
    const uint32_t lane_off = (uint32_t)((8 * (g >> 1) + (i16 >> 2)) * PPITCH + (16 * (g & 1) + 4 * (i16 & 3)) * 2);
    const uint32_t a_base = lane_off + (uint32_t)(wm * 128 * 2);
    const uint32_t b_base = (uint32_t)PR_OP + lane_off + (uint32_t)(wn * 32 * TN * 2);
    auto operand = [&](uint32_t addr) {
        const v4i16 lo = read_tr(addr);
        const v4i16 hi = read_tr(addr + 4 * PPITCH);
        typedef short v8i16 __attribute__((ext_vector_type(8)));
        const v8i16 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        return __builtin_bit_cast(bf16x8, v);
    };

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int t = 0; t < TN; ++t)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][t][v] = 0.0f;

#pragma unroll
    for (int c = 0; c < STAGES - 1; ++c)
        if (c_begin + c < c_end) issue(c_begin + c);
    for (int64_t chunk = c_begin; chunk < c_end; ++chunk) {
        // this wave's DMAs of stage `chunk` landed (later stages may still be in flight)
        const int later = (int)min(c_end - 1 - chunk, (int64_t)(STAGES - 2));
        wait_vmcnt(later * kDmas);
        __syncthreads();  // ... and every other wave's; all reads of stage chunk-1 are done
        if (chunk + STAGES - 1 < c_end) issue(chunk + STAGES - 1);  // into stage chunk-1's buffer
        const uint32_t st = smem_base + (uint32_t)((chunk % STAGES) * PR_STAGE);
        bf16x8 af[2][TM], bf[2][TN];
        auto load = [&](int u, int b) {
#pragma unroll
            for (int i = 0; i < TM; ++i) af[b][i] = operand(st + a_base + (uint32_t)(64 * i + u * 16 * PPITCH));
#pragma unroll
            for (int t = 0; t < TN; ++t) bf[b][t] = operand(st + b_base + (uint32_t)(64 * t + u * 16 * PPITCH));
        };
        load(0, 0);
#pragma unroll
        for (int u = 0; u < PIXR / 16; ++u) {
            if (u + 1 < PIXR / 16) load(u + 1, (u + 1) & 1);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int t = 0; t < TN; ++t) acc[i][t] = mfma32(af[u & 1][i], bf[u & 1][t], acc[i][t]);
        }
    }

    float* out = a.out + (int64_t)split * K * J;
    const int l32 = lane & 31, half = lane >> 5;
#pragma unroll
    for (int t = 0; t < TN; ++t) {
        const int col = j0 + wn * 32 * TN + 32 * t + l32;
        if (col >= J) continue;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int row = k0 + wm * 128 + 32 * i + 8 * (v >> 2) + 4 * half + (v & 3);
                if (row < K) {
                    float* o = out + (int64_t)row * J + col;
                    *o = a.accumulate ? *o + acc[i][t][v] : acc[i][t][v];
                }
            }
    }
}

}  // namespace

bool wgrad_dma_eligible(const WgradArgs& a) {
    const int64_t M = (int64_t)a.N * a.P * a.Q;
    const int64_t xbytes = (int64_t)a.N * a.H * a.W * a.C * 2;
    return a.C % 8 == 0 && a.K % 8 == 0 && M * a.K * 2 < 0x7FFFFFF0ll && xbytes < 0x7FFFFFF0ll;
}

WgradDmaPlan wgrad_dma_plan(int K, int J) {
    WgradDmaPlan p;
    // pixel-major rows for wide layers; the segment-major stages waste less of the
    // 256-row tile's copy work when K is narrow
    p.cfg = K >= 128 ? 1 : 0;
    const char* e = getenv("TBN_WGRAD_CFG");
    if (e && (atoi(e) == 0 || atoi(e) == 1)) p.cfg = atoi(e);
    p.tiles = ((K + TILE_K - 1) / TILE_K) * ((J + 255) / 256);
    p.resident_blocks = 256;  // one block per CU
    return p;
}

hipError_t launch_wgrad_dma(const WgradArgs& a, hipStream_t stream) {
    WgradDmaArgs ka;
    ka.a = a;
    ka.div_q = make_fastdiv((uint32_t)a.Q);
    ka.div_pq = make_fastdiv((uint32_t)a.P * (uint32_t)a.Q);
    const WgradDmaPlan p = wgrad_dma_plan(a.K, a.R * a.S * a.C);
    const dim3 grid((unsigned)(p.tiles * a.splits));
    if (p.cfg == 1)
        hipLaunchKernelGGL((wgrad_rows_kernel<64, 2>), grid, dim3(512), 0, stream, ka);
    else
        hipLaunchKernelGGL(wgrad_seg_kernel, grid, dim3(512), 0, stream, ka);
    return hipGetLastError();
}

}  // namespace tbn
