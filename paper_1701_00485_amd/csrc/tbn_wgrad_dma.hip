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
//   * stages of pixels in a ring of LDS buffers: the DMAs of later stages overlap the
//     MFMAs of the current one, and the operands of each 16-pixel step are read two steps
//     earlier (the pixel-major kernel; one step in the segment-major one);
//   * the pixel range is split over the grid (split-K): each split writes fp32 partials
//     that a second kernel adds in a fixed order (deterministic result).
// Two stage layouts:
//   * pixel-major (wide layers): each pixel's 256 dy channels / 256 x columns form one
//     512-byte row of the stage, two pixels per 1088-byte slot, so that one 64-lane DMA
//     instruction copies two pixels' contiguous bytes and the requests cover whole cache
//     lines; 48-pixel stages, three deep (an L2 prefetch of a later stage is an option);
//   * segment-major (K < 128): 64-pixel stages, two deep; for every 8-channel segment the
//     64 pixels' 16-byte pieces are contiguous (one DMA instruction, lane = pixel),
//     segments 1088 bytes apart; with few valid dy channels this issues fewer copies.
#include <cstdlib>
#include <type_traits>

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
    int32_t pf_dist;  // pixel-major kernel: stages between a copy and the L2 prefetch issued with it
};

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;

__device__ __forceinline__ v4i16 read_tr(uint32_t addr) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(uintptr_t)addr);
}

// Per-lane select by a wave-uniform 64-bit lane mask: bit i of `mask` set -> lane i gets
// `if_set`.  One v_cndmask with the mask in a scalar register pair.
__device__ __forceinline__ uint32_t lane_select(uint64_t mask, uint32_t if_clear, uint32_t if_set) {
    uint32_t r;
    asm("v_cndmask_b32_e64 %0, %1, %2, %3" : "=v"(r) : "v"(if_clear), "v"(if_set), "s"(mask));
    return r;
}

// 8 consecutive pixels of one channel as an MFMA operand (two transposing reads).
__device__ __forceinline__ bf16x8 operand(uint32_t addr) {
    const v4i16 lo = read_tr(addr);
    const v4i16 hi = read_tr(addr + 64);  // pixels + 4
    typedef short v8i16 __attribute__((ext_vector_type(8)));
    const v8i16 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    return __builtin_bit_cast(bf16x8, v);
}

// Instruction order of one 16-pixel step: its 8 MFMAs alternate with the 12 transposing
// reads of a later step's operands (two after each of the first four MFMAs, one after each
// of the others) and with the scalar work of the copy table, so that neither is issued in
// one burst (the reads spread this way measured ~6% faster than the compiler's own order
// on the 256 x 2304 training-layer gradient).
__device__ __forceinline__ void interleave_reads() {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // two LDS reads
        __builtin_amdgcn_sched_group_barrier(0x004, 8, 0);  // scalar work of the copy table
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x004, 8, 0);
    }
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
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < PIXS / 16; ++u) {
            if (u + 1 < PIXS / 16) load(u + 1, (u + 1) & 1);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int t = 0; t < TN; ++t) acc[i][t] = mfma32(af[u & 1][i], bf[u & 1][t], acc[i][t]);
            if (u + 1 < PIXS / 16) interleave_reads();
            __builtin_amdgcn_sched_barrier(0);
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
// then the same pixels of the x tile (256 columns).  Pixel rows are stored in pairs:
// pixels i and i + PIXR/2 of the stage share a 1088-byte slot (512 + 512 + 64 bytes of
// padding), so one DMA instruction with all 64 lanes active copies two pixels (each lane
// 16 bytes; the vector memory pipe issues a 32-lane copy at the cost of a full one) and
// every request covers whole 128-byte lines.  A transposing read touches four
// consecutive stage pixels and the four 8 further on (then the next four of each); in
// consecutive slots those rows start 64 bytes apart modulo 256, so every LDS bank is used
// at most twice.  The order in which the pixels enter the reduction follows this layout
// (a permutation within the stage).
constexpr int PP = 1088;  // bytes per pair of pixel rows

// PIXR pixels per stage (a multiple of 16), STAGES-deep ring; 2 x 4 waves of 128 x 64,
// two waves per SIMD.  (One wave per SIMD with 128 x 128 wave tiles reads a third less
// from LDS per MFMA but measured slower: the stage boundaries are no longer covered.)
// LIN: linear copy addressing (see below), chosen by the host.
template <int PIXR, int STAGES, bool PF, bool LIN>
__global__ __launch_bounds__(512, 1) void wgrad_rows_kernel(const WgradDmaArgs ka) {
    const WgradArgs& a = ka.a;
    constexpr int WAVES = 8;
    constexpr int WNW = 4;              // waves along j
    constexpr int TM = 4, TN = 2;       // wave tile 128 x 64 of the 256 x 256 block tile
    constexpr int NPAIR = PIXR / 2;     // pixel pairs per stage
    constexpr int PAIRS = NPAIR / WAVES;  // pairs each wave copies per stage
    constexpr int PR_OP = NPAIR * PP;   // one operand tile of a stage
    constexpr int PR_STAGE = 2 * PR_OP;
    constexpr int DUMP = STAGES * PR_STAGE;  // 256 bytes that the L2 prefetches land in
    static_assert(PIXR % 16 == 0 && NPAIR % WAVES == 0, "stage size");
    static_assert(DUMP + 256 <= 160 * 1024, "LDS");

    __shared__ __attribute__((aligned(1024))) uint8_t smem[DUMP + 256];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / WNW;
    const int wn = wave % WNW;

    const int K = a.K, C = a.C;
    const int J = a.R * a.S * C;
    const uint32_t PQ = (uint32_t)a.P * a.Q;
    const int64_t M = (int64_t)a.N * PQ;
    const int tilesJ = (J + 255) / 256;
    const int tiles = tilesJ * ((K + 255) / 256);
    const int t_ = (int)xcd_remap(blockIdx.x, gridDim.x);
    const int split = t_ / tiles;
    const int k0 = ((t_ % tiles) / tilesJ) * 256;
    const int j0 = ((t_ % tiles) % tilesJ) * 256;
    // this split's pixels (the ranges are given in 64-pixel chunks) and its stages
    const int64_t m_begin = (int64_t)split * a.chunks_per_split * 64;
    const int64_t m_end = min(m_begin + (int64_t)a.chunks_per_split * 64, M);
    const int nst = m_end > m_begin ? (int)((m_end - m_begin + PIXR - 1) / PIXR) : 0;

    const v4i rs_dy = make_rsrc(a.dy, (uint32_t)(M * K * 2));
    const v4i rs_x = make_rsrc(a.x, (uint32_t)((int64_t)a.N * a.H * a.W * C * 2));
    const uint32_t smem_base = lds_addr(smem);

    // this lane's 8-channel segment of the dy row and of the x column tile, and which
    // pixel of a pair it copies
    const int seg = lane & 31;
    const int half = lane >> 5;
    const bool dy_ok = k0 + 8 * seg < K;
    const uint32_t dy_col = (uint32_t)(k0 + 8 * seg) * 2u;
    const uint32_t dy_bad = dy_ok ? 0u : 0x80000000u;
    const int jx = j0 + 8 * seg;
    const bool x_ok = jx < J;
    const int rsx = x_ok ? jx / C : 0;
    const int xc = x_ok ? jx - rsx * C : 0;
    const int xr = rsx / a.S, xs = rsx - (rsx / a.S) * a.S;
    const uint32_t HWC = (uint32_t)((int64_t)a.H * a.W * C);

    // (image, h, w) of output pixel m, for the x tap (r, s)
    auto locate = [&](uint32_t mm, int r, int s_, uint32_t* img, int* h, int* w) {
        *img = fdiv(mm, ka.div_pq);
        const uint32_t pq = mm - *img * PQ;
        const uint32_t p = fdiv(pq, ka.div_q);
        const uint32_t q_ = pq - p * (uint32_t)a.Q;
        *h = (int)p * a.sh - a.ph + r;
        *w = (int)q_ * a.sw - a.pw + s_;
    };

    // Byte offsets of this lane's copies of a stage (bit 31 set: outside the image or past
    // the split's last pixel, the hardware returns zeros): pair jj of the wave holds stage
    // pixels PAIRS wave + jj and that + NPAIR.  Computed for the next stage while the
    // MFMAs of the current one run.
    uint32_t o_dy[PAIRS], o_x[PAIRS];
    // the PAIRS pixels of a lane are consecutive: the first is located by division, the
    // others step q (and carry into p and the image)
    const int q_step = a.sw, p_step = a.sh;
    auto table_general = [&](int st_i) {
        const int64_t m0 = m_begin + (int64_t)st_i * PIXR + PAIRS * wave + NPAIR * half;
        uint32_t mm = m0 < m_end ? (uint32_t)m0 : 0u;
        uint32_t img = fdiv(mm, ka.div_pq);
        const uint32_t pq = mm - img * PQ;
        uint32_t p = fdiv(pq, ka.div_q);
        uint32_t q_ = pq - p * (uint32_t)a.Q;
        int h = (int)p * a.sh - a.ph + xr, w = (int)q_ * a.sw - a.pw + xs;
#pragma unroll
        for (int jj = 0; jj < PAIRS; ++jj) {
            const bool mok = m0 + jj < m_end;
            const uint32_t mj = mm + jj;
            o_dy[jj] = mok ? (mj * (uint32_t)K * 2u + dy_col) | dy_bad : 0x80000000u;
            const bool ok = mok && x_ok && (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W;
            o_x[jj] = ok ? (img * HWC + (uint32_t)((h * a.W + w) * C + xc)) * 2u : 0x80000000u;
            if (jj + 1 < PAIRS) {  // next output pixel
                ++q_;
                w += q_step;
                if (q_ == (uint32_t)a.Q) {
                    q_ = 0;
                    w -= a.Q * q_step;
                    ++p;
                    h += p_step;
                    if (p == (uint32_t)a.P) {
                        p = 0;
                        h -= a.P * p_step;
                        ++img;
                    }
                }
            }
        }
    };
    // Linear copies: a stride-1 convolution whose output has the input's size (P = H,
    // Q = W) maps output pixel m and tap (r, s) to input pixel m + (r - ph) W + (s - pw),
    // and with C % 256 == 0 the 256 columns of a block share one tap.  Then both halves'
    // offsets are one wave-uniform pixel offset (the first pixel of the pair; the second
    // lies NPAIR pixels on) plus a per-lane constant, and only the validity of the two
    // pixels (inside the image for the tap, before the split's end) is tested, on the
    // scalar unit; per copy one add and one select remain on the vector unit.
    const int tap = j0 / (LIN ? C : 1);
    const int tr = tap / a.S, ts = tap - (tap / a.S) * a.S;  // the block's tap (linear copies)
    const uint32_t ldy = dy_col + (uint32_t)(half * NPAIR * K * 2);
    const uint32_t lx = (uint32_t)(seg * 16 + half * NPAIR * C * 2);
    const int32_t x_shift = ((tr - a.ph) * a.W + (ts - a.pw)) * C + (LIN ? j0 - tap * C : 0);
    const uint64_t dyok_lanes = __builtin_amdgcn_ballot_w64(dy_ok);
    const uint32_t oob = 0x80000000u;
    // The linear table is built in two parts: a vector pass in which lane i tests stage
    // pixel i (inside the split, and inside the image for the block's tap) and the wave
    // collects the answers as one 64-bit mask, then per pair a few scalar bit tests that
    // turn the mask bits of its two pixels into the lane masks of the selects.  The main
    // loop places the parts between the MFMAs of different steps.
    uint64_t xin = 0;  // bit i: stage pixel i is in the split and its tap inside the image
    auto table_linear_mask = [&](int st_i) {
        const int32_t s0 = (int32_t)m_begin + st_i * PIXR;  // first pixel of the stage (< 2^31)
        const int32_t ms = s0 + lane;
        const bool in = lane < PIXR && ms < (int32_t)m_end;
        const uint32_t mm = in ? (uint32_t)ms : 0u;
        const uint32_t pq = mm - fdiv(mm, ka.div_pq) * PQ;
        const uint32_t p = fdiv(pq, ka.div_q);
        const uint32_t q_ = pq - p * (uint32_t)a.Q;
        const bool inside = (unsigned)((int)p - a.ph + tr) < (unsigned)a.H &&
                            (unsigned)((int)q_ - a.pw + ts) < (unsigned)a.W;
        xin = __builtin_amdgcn_ballot_w64(in && inside);
    };
    auto table_linear_select = [&](int st_i) {
        const int32_t s0 = (int32_t)m_begin + st_i * PIXR;
        const int32_t rem = (int32_t)m_end - s0;  // pixels of the split from the stage's first on
        const int32_t mA0 = s0 + PAIRS * wave;
#pragma unroll
        for (int jj = 0; jj < PAIRS; ++jj) {
            // stage pixels of the pair: A (lanes 0-31) and B = A + NPAIR (lanes 32-63)
            const int iA = PAIRS * wave + jj, iB = iA + NPAIR;
            const uint64_t ld_ok = (iA < rem ? 0x00000000FFFFFFFFull : 0ull) | (iB < rem ? 0xFFFFFFFF00000000ull : 0ull);
            const uint64_t lx_ok = (((xin >> iA) & 1ull) ? 0x00000000FFFFFFFFull : 0ull) |
                                   (((xin >> iB) & 1ull) ? 0xFFFFFFFF00000000ull : 0ull);
            const uint32_t mj = (uint32_t)(mA0 + jj);  // wraps harmlessly where masked off
            o_dy[jj] = lane_select(ld_ok & dyok_lanes, oob, mj * (uint32_t)K * 2u + ldy);
            o_x[jj] = lane_select(lx_ok, oob, (mj * (uint32_t)C + (uint32_t)x_shift) * 2u + lx);
        }
    };
    auto table = [&](int st_i) {
        if constexpr (LIN) {
            table_linear_mask(st_i);
            table_linear_select(st_i);
        } else {
            table_general(st_i);
        }
    };
    // The table of stage Y is needed when Y is issued, two steps before the end of stage
    // Y - STAGES, and may be built once stage Y-1 has been issued.  In stage `it` the
    // linear table of stage it+STAGES+1 starts in the last step (the mask pass) and that of
    // stage it+STAGES is finished in the first step (the selects); with two steps per stage
    // all of it in the last step.  The general table is built whole in the last step.
    constexpr int NSTEP = PIXR / 16;
    auto table_part = [&](int it, int u) {
        if constexpr (LIN) {
            if (NSTEP == 2) {
                if (u == 1) table(it + STAGES + 1);
            } else {
                if (u == NSTEP - 1) table_linear_mask(it + STAGES + 1);
                if (u == 0) table_linear_select(it + STAGES);
            }
        } else {
            if (u == NSTEP - 1) table_general(it + STAGES + 1);
        }
    };
    int islot = 0;  // ring slot of the next stage to issue
    auto issue = [&](int) {
        const uint32_t st = smem_base + (uint32_t)(islot * PR_STAGE);
        islot = islot + 1 == STAGES ? 0 : islot + 1;
#pragma unroll
        for (int jj = 0; jj < PAIRS; ++jj) {
            const int j = PAIRS * wave + jj;  // pair slot (wave-uniform)
            dma_b128(rs_dy, st + (uint32_t)(j * PP), o_dy[jj]);
            dma_b128(rs_x, st + (uint32_t)(PR_OP + j * PP), o_x[jj]);
        }
    };
    constexpr int kDmas = 2 * PAIRS;

    // L2 prefetch of a later stage: one 4-byte copy per thread into a dump area touches one
    // 128-byte line (waves 0-3: the dy rows, stage pixel (tid % 256) / 4, line tid % 4 of
    // its 512 bytes; waves 4-7: the same for the x rows), so that the copies of that stage
    // find their lines in L2.
    const int pf_line = tid & 3;
    const int pf_pix = (tid & 255) >> 2;
    const bool pf_is_x = wave >= 4;  // wave-uniform
    const int pf_k = k0 + 64 * pf_line;
    const int pf_j = j0 + 64 * pf_line;
    const bool pf_jok = pf_j < J;
    const int pf_rs = pf_jok ? pf_j / C : 0;
    const int pf_c = pf_jok ? pf_j - pf_rs * C : 0;
    const int pf_r = pf_rs / a.S, pf_s = pf_rs - (pf_rs / a.S) * a.S;
    auto prefetch = [&](int st_i) {
        const int64_t m = m_begin + (int64_t)st_i * PIXR + pf_pix;
        const bool mok = pf_pix < PIXR && m < m_end;
        const uint32_t mm = mok ? (uint32_t)m : 0u;
        if (pf_is_x) {
            uint32_t img;
            int h, w;
            locate(mm, pf_r, pf_s, &img, &h, &w);
            const bool ok = mok && pf_jok && (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W;
            dma_b32(rs_x, smem_base + DUMP,
                    ok ? (img * HWC + (uint32_t)((h * a.W + w) * C + pf_c)) * 2u : 0x80000000u);
        } else {
            dma_b32(rs_dy, smem_base + DUMP,
                    mok && pf_k < K ? (mm * (uint32_t)K + (uint32_t)pf_k) * 2u : 0x80000000u);
        }
    };
    const int pf_dist = ka.pf_dist;

    // transposing reads: lane (g = lane / 16, i = lane % 16) reads the 8 bytes of channels
    // 16 (g % 2) + 4 (i % 4) .. + 3 of stage pixel 16 u + 8 (g / 2) + i / 4 (+ 4 for the
    // second read) in step u; stage pixel r sits at (r % NPAIR) * PP + (r / NPAIR) * 512.
    // One address register per (ring slot, step, operand), masked to the LDS size so that
    // the compiler can prove it non-negative and fold the constant offsets of the other
    // rows of the wave tile into the read instructions.
    constexpr int NU = PIXR / 16;
    const int g = lane >> 4, i16 = lane & 15;
    const int rho = 8 * (g >> 1) + (i16 >> 2);
    const uint32_t col_off = (uint32_t)((16 * (g & 1) + 4 * (i16 & 3)) * 2);
    const uint32_t a_base = (uint32_t)(wm * 128 * 2);
    const uint32_t b_base = (uint32_t)PR_OP + (uint32_t)(wn * 32 * TN * 2);
    uint32_t ra[STAGES][NU], rb[STAGES][NU];
#pragma unroll
    for (int sl = 0; sl < STAGES; ++sl)
#pragma unroll
        for (int u = 0; u < NU; ++u) {
            const int r = 16 * u + rho;
            const uint32_t ro = (uint32_t)((r % NPAIR) * PP + (r / NPAIR) * 512) + col_off;
            ra[sl][u] = (smem_base + (uint32_t)(sl * PR_STAGE) + a_base + ro) & 0x3FFFFu;
            rb[sl][u] = (smem_base + (uint32_t)(sl * PR_STAGE) + b_base + ro) & 0x3FFFFu;
        }
    auto operand = [&](uint32_t addr) {
        const v4i16 lo = read_tr(addr);
        const v4i16 hi = read_tr(addr + 4 * PP);
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

    // Pipeline: every ring slot is filled in the prologue; stage `it` is multiplied step by
    // step with the operands of each step read two steps earlier.  Two steps before the end
    // of stage `it` a barrier certifies that every wave is done reading stage `it` (the
    // operands of its last two steps are already in registers) and that stage it+1 has
    // landed; the copies of stage it + STAGES then go into stage it's slot, and the last
    // two steps' MFMAs overlap the copies and the reads of stage it+1's first two steps.
    // So no wave waits on LDS reads at a stage boundary, and every read has a whole step
    // of MFMAs to complete.  With PF every issue() is followed by one prefetch; a stage's
    // copies are complete once at most the copies (and prefetches) issued after them are
    // outstanding.
#pragma unroll
    for (int c = 0; c < STAGES; ++c) {
        table(c);
        if (c < nst) {
            issue(c);
            if constexpr (PF) prefetch(c + pf_dist);
        }
    }
    table(STAGES);
    // wait until stage x's copies landed, with the copies of the `later` stages issued after
    // it (stages x+1 .. x+later) still allowed in flight; where fewer than that were issued
    // (the last stages), wait for everything
    auto wait_stage = [&](int x, auto later_c) {
        constexpr int later = decltype(later_c)::value;
        if (x + later < nst)
            wait_vmcnt(PF ? later * (kDmas + 1) + 1 : later * kDmas);
        else
            wait_vmcnt(0);
    };
    // in the order the MFMAs use them (row 0 with every column first), so that the first
    // MFMAs of a step wait only for the reads issued earliest
    auto load = [&](int sl, int u, bf16x8* af, bf16x8* bf) {
        af[0] = operand(ra[sl][u]);
#pragma unroll
        for (int t = 0; t < TN; ++t) bf[t] = operand(rb[sl][u] + (uint32_t)(64 * t));
#pragma unroll
        for (int i = 1; i < TM; ++i) af[i] = operand(ra[sl][u] + (uint32_t)(64 * i));
    };
    bf16x8 af[TM], bf[TN];    // operands of the next step to multiply
    bf16x8 af1[TM], bf1[TN];  // ... and of the step after it
    if (nst > 0) {
        wait_stage(0, std::integral_constant<int, STAGES - 1>{});  // stages 0 .. STAGES-1 issued
        __syncthreads();
        load(0, 0, af, bf);
        load(0, 1, af1, bf1);
    }
    // one stage, in ring slot SL (a compile-time constant: the loop below is unrolled over
    // the ring)
    auto stage = [&](int it, auto slot) {
        constexpr int SL = decltype(slot)::value;
        constexpr int SN = SL + 1 == STAGES ? 0 : SL + 1;
#pragma unroll
        for (int u = 0; u < NSTEP; ++u) {
            bf16x8 naf[TM], nbf[TN];  // operands of step u + 2
            if (u + 2 < NSTEP) {
                load(SL, u + 2, naf, nbf);
            } else {
                if (u + 2 == NSTEP) {
                    // stage it+1 landed (this wave's copies, then every wave's) and every
                    // wave is done reading stage it
                    wait_stage(it + 1, std::integral_constant<int, STAGES - 2>{});  // 0 .. it+STAGES-1 issued
                    __syncthreads();
                }
                load(SN, u + 2 - NSTEP, naf, nbf);  // unused after the last stage
            }
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int t = 0; t < TN; ++t) acc[i][t] = mfma32(af[i], bf[t], acc[i][t]);
            // the copies of stage it + STAGES into stage it's slot, behind the MFMAs of the
            // step that follows the barrier
            if (u + 2 == NSTEP && it + STAGES < nst) {
                issue(it + STAGES);
                if constexpr (PF) prefetch(it + STAGES + pf_dist);
            }
            // copy offsets between the MFMAs (harmless past the last stage: nothing issues
            // them)
            table_part(it, u);
            interleave_reads();
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                af[i] = af1[i];
                af1[i] = naf[i];
            }
#pragma unroll
            for (int t = 0; t < TN; ++t) {
                bf[t] = bf1[t];
                bf1[t] = nbf[t];
            }
        }
    };
    for (int it = 0; it < nst; it += STAGES) {
        stage(it, std::integral_constant<int, 0>{});
        if constexpr (STAGES > 1)
            if (it + 1 < nst) stage(it + 1, std::integral_constant<int, 1>{});
        if constexpr (STAGES > 2)
            if (it + 2 < nst) stage(it + 2, std::integral_constant<int, 2>{});
        if constexpr (STAGES > 3)
            if (it + 3 < nst) stage(it + 3, std::integral_constant<int, 3>{});
    }
    static_assert(STAGES <= 4, "ring unrolled up to four slots");

    float* out = a.out + (int64_t)split * K * J;
    const int l32 = lane & 31;
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
    const int forced = knob(KNOB_WGRAD_CFG);
    if (forced == 0 || forced == 1) p.cfg = forced;
    p.tiles = ((K + TILE_K - 1) / TILE_K) * ((J + 255) / 256);
    p.resident_blocks = 256;  // one block per CU
    // pixel-major kernel: 48-pixel stages in a three-deep ring (measured best of 32 / 48 / 64)
    p.pix = 48;
    const int px = knob(KNOB_WGRAD_PIX);
    if (px == 32 || px == 64) p.pix = px;
    return p;
}

template <bool LIN>
static void launch_rows(int pix, bool pf, dim3 grid, const WgradDmaArgs& ka, hipStream_t stream) {
    switch (pix) {
        case 32: hipLaunchKernelGGL((wgrad_rows_kernel<32, 4, false, LIN>), grid, dim3(512), 0, stream, ka); break;
        case 64: hipLaunchKernelGGL((wgrad_rows_kernel<64, 2, false, LIN>), grid, dim3(512), 0, stream, ka); break;
        default:
            if (pf)
                hipLaunchKernelGGL((wgrad_rows_kernel<48, 3, true, LIN>), grid, dim3(512), 0, stream, ka);
            else
                hipLaunchKernelGGL((wgrad_rows_kernel<48, 3, false, LIN>), grid, dim3(512), 0, stream, ka);
            break;
    }
}

hipError_t launch_wgrad_dma(const WgradArgs& a, hipStream_t stream) {
    WgradDmaArgs ka;
    ka.a = a;
    ka.div_q = make_fastdiv((uint32_t)a.Q);
    ka.div_pq = make_fastdiv((uint32_t)a.P * (uint32_t)a.Q);
    // L2 prefetch of a later stage: off by default (measured ~9% slower on the training
    // layer once the reads and MFMAs are interleaved); the prefetch knob (stages ahead)
    // turns it on
    const int pf = knob(KNOB_WGRAD_PF);
    ka.pf_dist = pf > 0 ? pf : 0;
    const WgradDmaPlan p = wgrad_dma_plan(a.K, a.R * a.S * a.C);
    const dim3 grid((unsigned)(p.tiles * a.splits));
    if (p.cfg == 1) {
        // linear copy addressing: stride 1, output the input's size, whole 256-column
        // blocks of one tap
        const bool lin = a.sh == 1 && a.sw == 1 && a.P == a.H && a.Q == a.W && a.C % 256 == 0;
        if (lin)
            launch_rows<true>(p.pix, ka.pf_dist > 0, grid, ka, stream);
        else
            launch_rows<false>(p.pix, ka.pf_dist > 0, grid, ka, stream);
    } else {
        hipLaunchKernelGGL(wgrad_seg_kernel, grid, dim3(512), 0, stream, ka);
    }
    return hipGetLastError();
}

}  // namespace tbn
