// tbn_wgrad_dma.hip -- gradient with respect to the approximate filter (Algorithm 1,
// backward step; Sec. 3 applies it unchanged to the real weights):
//     dW[k][j] = sum_m dy[m][k] * x_col[m][j],   m = (n,p,q) output pixel, j = (r,s,c),
// for bf16 activations with C % 8 == 0 and K % 8 == 0.
//
// Both operands arrive with the reduction index (the pixel) outermost, while the MFMA
// wants 8 consecutive reduction elements per lane.  Instead of transposing in registers,
// the kernel copies the raw tiles into LDS with LDS-DMA buffer loads and forms the MFMA
// operands with the gfx950 transposing LDS read (ds_read_b64_tr_b16: a 16-lane group
// turns a 16 x 4 block of 16-bit values into 4 consecutive rows per lane), so the main
// loop spends no vector ALU work on data movement:
//   * a block of 8 waves owns a 256 (k) x 256 (j) output tile; each wave 128 x 64 made of
//     32x32 v_mfma_f32_32x32x16_bf16 tiles with fp32 accumulators;
//   * a stage is 64 pixels.  Each operand tile of a stage is stored segment-major: for
//     every 8-channel segment, the 64 pixels' 16-byte pieces are contiguous (exactly one
//     DMA instruction, lane = pixel), and the segments are 1088 bytes apart so that the
//     transposing reads of two neighbouring segments hit different banks;
//   * lane = pixel for every DMA, so a lane decomposes one pixel per stage; the tap
//     (r, s, c) of an x segment is wave-uniform;
//   * the pixel range is split over the grid (split-K): each split writes fp32 partials
//     that a second kernel adds in a fixed order (deterministic result);
//   * two LDS stages (136 KiB): the DMAs of stage c+1 overlap the MFMAs of stage c.
#include "tbn_device.h"
#include "tbn_dma.h"
#include "tbn_kernels.h"

namespace tbn {

namespace {

constexpr int PIX = 64;              // pixels per stage
constexpr int SEGS = 32;             // 8-channel segments per operand tile (256 channels)
constexpr int SEG_PITCH = 64 * 16 + 64;
constexpr int OP_BYTES = SEGS * SEG_PITCH;
constexpr int STAGE_BYTES = 2 * OP_BYTES;  // dy tile then x tile
constexpr int TILE = 256;

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

__global__ __launch_bounds__(512, 1) void wgrad_dma_kernel(const WgradDmaArgs ka) {
    const WgradArgs& a = ka.a;
    constexpr int TM = 4, TN = 2;  // wave tile 128 x 64

    __shared__ __attribute__((aligned(1024))) uint8_t smem[2 * STAGE_BYTES];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 2;  // 0..1
    const int wn = wave & 3;   // 0..3

    const int K = a.K, C = a.C;
    const int J = a.R * a.S * C;
    const uint32_t PQ = (uint32_t)a.P * a.Q;
    const int64_t M = (int64_t)a.N * PQ;
    const int64_t nchunks = (M + PIX - 1) / PIX;
    const int tilesJ = (J + TILE - 1) / TILE;
    const int tiles = tilesJ * ((K + TILE - 1) / TILE);
    const int t_ = (int)xcd_remap(blockIdx.x, gridDim.x);
    const int split = t_ / tiles;
    const int k0 = ((t_ % tiles) / tilesJ) * TILE;
    const int j0 = ((t_ % tiles) % tilesJ) * TILE;
    const int64_t c_begin = (int64_t)split * a.chunks_per_split;
    const int64_t c_end = min(c_begin + (int64_t)a.chunks_per_split, nchunks);

    const v4i rs_dy = make_rsrc(a.dy, (uint32_t)(M * K * 2));
    const v4i rs_x = make_rsrc(a.x, (uint32_t)((int64_t)a.N * a.H * a.W * C * 2));
    const uint32_t smem_base = lds_addr(smem);

    // segments this wave copies: 4 of dy (channels k0 + 8 sg) and 4 of x (columns j0 + 8 sg)
    int xr[4], xs[4], xc[4];
    bool dy_ok[4], x_ok[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int sg = 4 * wave + q;
        dy_ok[q] = k0 + 8 * sg < K;
        const int j = j0 + 8 * sg;
        x_ok[q] = j < J;
        const int rs = x_ok[q] ? j / C : 0;
        xc[q] = x_ok[q] ? j - rs * C : 0;
        xr[q] = rs / a.S;
        xs[q] = rs - xr[q] * a.S;
    }
    const int64_t HWC = (int64_t)a.H * a.W * C;

    auto issue = [&](int64_t chunk) {
        const uint32_t st = smem_base + (uint32_t)((chunk & 1) * STAGE_BYTES);
        const int64_t m = chunk * PIX + lane;
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
        for (int q = 0; q < 4; ++q) {
            const int sg = 4 * wave + q;
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

    if (c_begin < c_end) issue(c_begin);
    for (int64_t chunk = c_begin; chunk < c_end; ++chunk) {
        wait_vmcnt(0);    // this wave's DMAs of stage `chunk` landed
        __syncthreads();  // ... and every other wave's; all reads of the other buffer are done
        if (chunk + 1 < c_end) issue(chunk + 1);
        const uint32_t st = smem_base + (uint32_t)((chunk & 1) * STAGE_BYTES);
#pragma unroll
        for (int u = 0; u < 4; ++u) {  // 16 pixels per MFMA step
            bf16x8 af[TM], bf[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i) af[i] = operand(st + a_base + (uint32_t)(4 * i * SEG_PITCH + u * 256));
#pragma unroll
            for (int t = 0; t < TN; ++t) bf[t] = operand(st + b_base + (uint32_t)(4 * t * SEG_PITCH + u * 256));
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int t = 0; t < TN; ++t) acc[i][t] = mfma32(af[i], bf[t], acc[i][t]);
        }
    }

    float* out = a.out + (int64_t)split * K * J;
    const int l32 = lane & 31, half = lane >> 5;
#pragma unroll
    for (int t = 0; t < TN; ++t) {
        const int col = j0 + wn * 64 + 32 * t + l32;
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

int wgrad_dma_tiles(int K, int J) { return ((K + TILE - 1) / TILE) * ((J + TILE - 1) / TILE); }

hipError_t launch_wgrad_dma(const WgradArgs& a, hipStream_t stream) {
    WgradDmaArgs ka;
    ka.a = a;
    ka.div_q = make_fastdiv((uint32_t)a.Q);
    ka.div_pq = make_fastdiv((uint32_t)a.P * (uint32_t)a.Q);
    const int tiles = wgrad_dma_tiles(a.K, a.R * a.S * a.C);
    hipLaunchKernelGGL(wgrad_dma_kernel, dim3((unsigned)(tiles * a.splits)), dim3(512), 0, stream, ka);
    return hipGetLastError();
}

}  // namespace tbn
