// tbn_conv_dma.hip -- the main implicit-GEMM convolution kernel for bf16 NHWC activations
// with C % 8 == 0 (every layer of the workloads except the C = 1 / C = 3 first layers).
// It computes the same GEMM as tbn_conv.hip (the forward pass, Sec. 2 Eq. 1, and the
// backward-data pass through the approximate filters, Sec. 3) at a much lower
// instruction count per MFMA:
//
//   * every operand of a stage goes from memory straight into LDS with buffer loads in
//     LDS-DMA mode: the activation tile (16 bytes per lane), the 1 KiB packed-code blocks
//     of the tile's filters, and in the backward-data pass the stage's bf16 scale pairs.
//     Zero padding costs nothing: an out-of-image tap gets an out-of-range buffer offset
//     and the hardware returns zeros.  Which of a row's R*S taps fall inside the image is
//     precomputed once per row as a 64-bit mask;
//   * the DMAs run up to three stages deep (a ring of LDS buffers): the loads of stage
//     c+2 are in flight while stage c is multiplied.  They are issued from inline
//     assembly and waited for with explicit vmcnt counts, because the compiler treats
//     any LDS-DMA as a write to all of LDS and would otherwise wait for every
//     outstanding DMA before each LDS read;
//   * LDS rows are 128 bytes (64 bf16) with the 16-byte segments XOR-swizzled by
//     (row / 2) % 8, so the DMA writes and the 16-byte MFMA operand reads are free of
//     bank conflicts without padding;
//   * the two-bit filter operand is decoded in registers from the LDS copy of the codes
//     (one AND and one shift-add per bf16 pair, per-lane masks precomputed);
//   * the MFMA is issued with the decoded filters as its first operand, so the
//     accumulators hold the transposed tile and each lane owns runs of four consecutive
//     output channels of one pixel; the epilogue stages each tile row through LDS with
//     16-byte writes and applies scale, bias, residual and ReLU to 8 consecutive
//     channels per lane, written with 16-byte stores;
//   * blocks are ordered XCD-aware (each XCD runs a contiguous range of tiles).
//
// M0 is written by the DMA helper; nothing else in these kernels uses M0.
#include "tbn_device.h"
#include "tbn_dma.h"
#include "tbn_kernels.h"

namespace tbn {

namespace {

constexpr int BK = 64;     // reduction elements per stage
constexpr int ROWB = 128;  // LDS bytes per activation row of a stage

template <int BM, int BN>
struct StageLayout {
    static constexpr int A = 0;                  // BM rows x 128 B
    static constexpr int B = BM * ROWB;          // BN filters x 16 B (BN/64 blocks of 1 KiB)
    static constexpr int P = B + BN * 16;        // 256 B of bf16 scale pairs (backward-data)
    static constexpr int BYTES = P + 256;
};

// Sum of the split-K partials of outputs (row, col0 .. col0 + 7) in split order, then the
// epilogue (partial rows are Kp = round_up(Kf, 8) wide; columns past Kf are skipped).  The
// column factors and the residual are loaded first, then the partials eight splits at a
// time (the last batch masked, its missing terms zero), so that a thread waits for memory
// about once per eight splits rather than once per split of the tail.
__device__ __forceinline__ void split_epilogue_group(const ConvGemmArgs& a, int64_t M, int64_t row, int col0) {
    const int Kf = a.Kf;
    const int Kp = (Kf + 7) & ~7;
    const int64_t po = row * Kp + col0;
    const int64_t o = row * Kf + col0;
    const bool full = col0 + 8 <= Kf;  // all 8 columns real (always when Kf % 8 == 0)
    float sc[8], bi[8], rs[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const int col = col0 + e < Kf ? col0 + e : Kf - 1;  // past Kf: computed, never stored
        sc[e] = a.colscale ? a.colscale[col] : 1.0f;
        if (a.scale) sc[e] *= a.scale[col];
        bi[e] = a.bias ? a.bias[col] : 0.0f;
        rs[e] = 0.0f;
    }
    if (a.residual) {
        if (a.y_f32) {
            const float* rp = reinterpret_cast<const float*>(a.residual) + o;
#pragma unroll
            for (int e = 0; e < 8; ++e)
                if (col0 + e < Kf) rs[e] = rp[e];
        } else if (full && (Kf % 8) == 0) {
            const u32x4 r8 = *reinterpret_cast<const u32x4*>(reinterpret_cast<const uint16_t*>(a.residual) + o);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                rs[2 * e] = bf16_bits_to_f32(r8[e] & 0xFFFFu);
                rs[2 * e + 1] = bf16_bits_to_f32(r8[e] >> 16);
            }
        } else {
            const uint16_t* rp = reinterpret_cast<const uint16_t*>(a.residual) + o;
#pragma unroll
            for (int e = 0; e < 8; ++e)
                if (col0 + e < Kf) rs[e] = bf16_bits_to_f32(rp[e]);
        }
    }
    float v8[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int z = 0; z < a.splits; z += 8) {
        f32x4 lo[8], hi[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            lo[u] = hi[u] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
            if (z + u < a.splits) {
                const float* pp = a.partial + (int64_t)(z + u) * M * Kp + po;
                lo[u] = *reinterpret_cast<const f32x4*>(pp);
                hi[u] = *reinterpret_cast<const f32x4*>(pp + 4);
            }
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            v8[0] += lo[u].x; v8[1] += lo[u].y; v8[2] += lo[u].z; v8[3] += lo[u].w;
            v8[4] += hi[u].x; v8[5] += hi[u].y; v8[6] += hi[u].z; v8[7] += hi[u].w;
        }
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) v8[e] = v8[e] * sc[e] + bi[e] + rs[e];
    if (a.relu) {
#pragma unroll
        for (int e = 0; e < 8; ++e) v8[e] = fmaxf(v8[e], 0.0f);
    }
    if ((Kf % 8) == 0) {
        if (a.y_f32) {
            float* yp = reinterpret_cast<float*>(a.y) + o;
            *reinterpret_cast<f32x4*>(yp) = f32x4{v8[0], v8[1], v8[2], v8[3]};
            *reinterpret_cast<f32x4*>(yp + 4) = f32x4{v8[4], v8[5], v8[6], v8[7]};
        } else {
            *reinterpret_cast<u32x4*>(reinterpret_cast<uint16_t*>(a.y) + o) =
                u32x4{pack_bf16x2(v8[0], v8[1]), pack_bf16x2(v8[2], v8[3]), pack_bf16x2(v8[4], v8[5]),
                      pack_bf16x2(v8[6], v8[7])};
        }
    } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            if (col0 + e >= Kf) break;
            if (a.y_f32)
                reinterpret_cast<float*>(a.y)[o + e] = v8[e];
            else
                reinterpret_cast<uint16_t*>(a.y)[o + e] = (uint16_t)f32_to_bf16_bits(v8[e]);
        }
    }
}

// UNI: C % 64 == 0, so all 64 elements of a stage share one tap (r, s) and the tap
// bookkeeping is wave-uniform (scalar registers).
// Tiles of 256 x 256 run one block per CU (one wave per SIMD, 128 x 128 accumulators each);
// smaller tiles two.
// G > 1: the block is G groups of four waves; group g reduces its own contiguous range of
// the tile's stages with its own LDS ring (the grid's reduction split s covers ranges
// s G .. s G + G - 1), and at the end groups 1 .. G-1 hand their sums to group 0 through
// LDS, which adds them in group order and runs the epilogue.  This gives a tile G waves
// per SIMD where the grid has too few tiles for two blocks per CU, without partial sums in
// memory or a second kernel.
template <int BM, int BN, int WAVES_M, int WAVES_N, int STAGES, bool BWD, bool UNI, int G>
__global__ __launch_bounds__(256 * G, (BM * BN >= 65536 || G > 1) ? 1 : 2) void conv_dma_kernel(const ConvGemmArgs a) {
    constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
    constexpr int TM = WM / 32, TN = WN / 32;
    constexpr int AR = BM / 32;      // activation DMAs per wave per stage (8 rows each)
    constexpr int NBLK = BN / 64;    // 1 KiB code blocks per stage
    using L = StageLayout<BM, BN>;
    static_assert(WAVES_M * WAVES_N == 4, "four waves per block");
    static_assert(TM >= 1 && TN >= 1 && BM % 32 == 0 && BN % 64 == 0 && NBLK <= 4, "tile shape");
    static_assert(STAGES * L::BYTES >= 4 * 32 * (WN + 4) * 4, "epilogue staging fits in the ring");
    // G > 1: the sums of groups 1 .. G-1 are handed over behind group 0's epilogue staging
    constexpr int NACC = TM * TN * 16;  // accumulators per lane
    constexpr int XOFF = ((4 * 32 * (WN + 4) * 4 + 1023) / 1024) * 1024;
    static_assert(G == 1 || G * STAGES * L::BYTES >= XOFF + (G - 1) * 256 * NACC * 4, "group sums fit in LDS");

    __shared__ __attribute__((aligned(1024))) uint8_t smem[G * STAGES * L::BYTES];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int grp = G > 1 ? __builtin_amdgcn_readfirstlane(tid >> 8) : 0;  // group of four waves
    const int wave = __builtin_amdgcn_readfirstlane((tid >> 6) & 3);     // wave within the group
    const int wm = wave / WAVES_N;
    const int wn = wave % WAVES_N;
    const int half = lane >> 5;
    const int l32 = lane & 31;

    const int64_t PQ = (int64_t)a.P * a.Q;
    const int64_t M = (int64_t)a.N * PQ;
    const int C = a.C;
    const int n = a.R * a.S * C;
    const int nchunks = (n + BK - 1) / BK;
    const int KB = (a.Kf + 63) / 64;
    const uint32_t tilesN = (uint32_t)(a.Kf + BN - 1) / BN;
    const uint32_t tiles = (uint32_t)((M + BM - 1) / BM) * tilesN;
    // XCD-aware order over (split, tile); each split reduces a contiguous range of stages.
    // Block counts are below 2^31 (checked by the host), so 32-bit magic-number divisions.
    const uint32_t work = (uint32_t)xcd_remap(blockIdx.x, gridDim.x);
    const int split = (int)fdiv(work, a.div_tiles);
    const uint32_t tile = work - (uint32_t)split * tiles;
    const uint32_t mtile = fdiv(tile, a.div_tilesN);
    const int64_t m0 = (int64_t)mtile * BM;
    const int n0 = (int)(tile - mtile * tilesN) * BN;
    const int c_begin = (split * G + grp) * a.chunks_per_split;
    const int c_end = min(c_begin + a.chunks_per_split, nchunks);
    const int nloc = max(c_end - c_begin, 0);
    // every group runs the same number of iterations (and barriers); a group whose range is
    // shorter skips the copies and MFMAs of the missing stages
    const int niter = G > 1 ? a.chunks_per_split : nloc;

    const v4i rs_x = make_rsrc(a.x, (uint32_t)((int64_t)a.N * a.H * a.W * C * 2));
    const v4i rs_c = make_rsrc(a.codes, (uint32_t)((int64_t)KB * nchunks * 1024));
    v4i rs_p = rs_c;
    if constexpr (BWD) rs_p = make_rsrc(a.apair, (uint32_t)nchunks * 128u);
    uint8_t* const ring = smem + grp * (STAGES * L::BYTES);  // this group's LDS ring
    const uint32_t smem_base = lds_addr(ring);

    // ---- activation rows this lane fills: row = 8 * (wave + 4 j) + lane / 8 ----
    int32_t rbase[AR];      // element offset of the row's (h0, w0) in x (may be negative)
    uint32_t rmask[AR][2];  // bit r*S + s of the 64 set iff tap (r, s) lies inside the image
#pragma unroll
    for (int j = 0; j < AR; ++j) {
        const int64_t m = m0 + 8 * (wave + 4 * j) + (lane >> 3);
        uint64_t mask = 0;
        rbase[j] = 0;
        if (m < M) {
            const uint32_t mm = (uint32_t)m;  // < 2^31, checked by the host
            const uint32_t img = fdiv(mm, a.div_pq);
            const uint32_t pq = mm - img * (uint32_t)PQ;
            const uint32_t p = fdiv(pq, a.div_q);
            const uint32_t q = pq - p * (uint32_t)a.Q;
            const int h0 = (int)p * a.sh - a.ph, w0 = (int)q * a.sw - a.pw;
            rbase[j] = ((int32_t)img * a.H + h0) * a.W * C + w0 * C;
            // in-image taps: s in [slo, shi), r in [rlo, rhi); the row's bits wbits
            // replicated at every in-image r by one multiplication with the pattern
            // sum_r 2^(r*S) (its groups of S bits never overlap, R*S <= 63)
            const int slo = max(0, -w0), shi = min(a.S, a.W - w0);
            const int rlo = max(0, -h0), rhi = min(a.R, a.H - h0);
            if (shi > slo && rhi > rlo) {
                const uint64_t wbits = (1ull << shi) - (1ull << slo);
                const uint64_t rowsel = (1ull << (rhi * a.S)) - (1ull << (rlo * a.S));
                const uint64_t rep = ((uint64_t)a.rep_hi << 32) | a.rep_lo;
                mask = wbits * (rep & rowsel);
            }
        }
        rmask[j][0] = (uint32_t)mask;
        rmask[j][1] = (uint32_t)(mask >> 32);
    }
    // logical 16-byte segment this lane loads (its LDS slot is lane % 8 of the row)
    const int lseg = (lane & 7) ^ ((4 * (wave & 1)) | ((lane >> 4) & 3));
    // general path: (r, s, c) of element 8 * lseg of the next stage to issue (per lane)
    int er = 0, es = 0, ec = 0;
    // uniform path: (r, s) and first channel of the next stage (the same for every lane)
    int ur = 0, us = 0, uc = 0;
    // uniform path, kept incrementally: utap = r * S + s, utoff2 = byte offset of (r, s, c0)
    // relative to a row's (h0, w0) = 2 * ((r * W + s) * C + c0)
    int utap = 0;
    uint32_t utoff2 = 0;
    uint32_t rb2s[AR];      // uniform path: byte offset of the row plus this lane's segment
    uint32_t nmask[AR][2];  // uniform path: complement of rmask (bit set = tap outside)
    if constexpr (UNI) {
#pragma unroll
        for (int j = 0; j < AR; ++j) {
            rb2s[j] = (uint32_t)(rbase[j] + 8 * lseg) << 1;
            nmask[j][0] = ~rmask[j][0];
            nmask[j][1] = ~rmask[j][1];
        }
        if (c_begin != 0) {  // a later reduction split: its first (r, s, c)
            const int e0 = c_begin * BK;
            const int rs = e0 / C;
            uc = e0 - rs * C;
            ur = rs / a.S;
            us = rs - ur * a.S;
            utap = rs;
            utoff2 = (uint32_t)((ur * a.W + us) * C + uc) << 1;
        }
    } else {
        const int e0 = c_begin * BK + lseg * 8;
        const int rs = e0 / C;
        ec = e0 - rs * C;
        er = rs / a.S;
        es = rs - er * a.S;
    }
    // code block of this wave: wave w copies the 1 KiB block w % NBLK of each stage (with
    // fewer than four blocks some waves copy the same block into the same place, identical
    // bytes), so that every wave issues the same number of DMAs per stage and the waits
    // below are compile-time counts
    const int cblk = wave % NBLK;
    const int fb = n0 / 64 + cblk;
    const bool codes_valid = fb < KB;
    constexpr int DMAS = AR + 1 + (BWD ? 1 : 0);  // per stage, every wave

    const uint32_t row_step2 = (uint32_t)((a.W - a.S) * C) << 1;  // next filter row, in bytes
    int islot = 0;  // ring slot of the next stage to issue
    auto issue = [&](int chunk) {
        const uint32_t st = smem_base + (uint32_t)(islot * L::BYTES);
        islot = islot + 1 == STAGES ? 0 : islot + 1;
        if constexpr (UNI) {
            // out-of-image taps (and the padding stage past the filter, tap clamped to
            // bit 63, which is clear in rmask because R*S <= 63) get offset bit 31 set,
            // beyond the buffer, so the hardware returns zeros
            const int tap = min(utap, 63);
            if (tap < 32) {
#pragma unroll
                for (int j = 0; j < AR; ++j) {
                    const uint32_t out = (nmask[j][0] << (31 - tap)) & 0x80000000u;
                    dma_b128(rs_x, st + L::A + (uint32_t)(8 * (wave + 4 * j) * ROWB), (rb2s[j] + utoff2) | out);
                }
            } else {
#pragma unroll
                for (int j = 0; j < AR; ++j) {
                    const uint32_t out = (nmask[j][1] << (63 - tap)) & 0x80000000u;
                    dma_b128(rs_x, st + L::A + (uint32_t)(8 * (wave + 4 * j) * ROWB), (rb2s[j] + utoff2) | out);
                }
            }
            // next stage: 64 channels on; past the last channel the next tap (s + 1), past
            // the last tap of a filter row the first tap of the next row
            uc += BK;
            utoff2 += 2 * BK;
            if (uc == C) {
                uc = 0;
                ++utap;
                if (++us == a.S) {
                    us = 0;
                    utoff2 += row_step2;
                }
            }
        } else {
            // taps past the filter (padding elements of the last stage) clamp to bit 63,
            // which is clear because R*S <= 63
            const int tap = min(er * a.S + es, 63);
            const int tword = tap >> 5, tbit = tap & 31;
            const int32_t toff = (er * a.W + es) * C + ec;
#pragma unroll
            for (int j = 0; j < AR; ++j) {
                const bool ok = ((tword ? rmask[j][1] : rmask[j][0]) >> tbit) & 1u;
                const uint32_t off = ok ? (uint32_t)(rbase[j] + toff) << 1 : 0x80000000u;
                dma_b128(rs_x, st + L::A + (uint32_t)(8 * (wave + 4 * j) * ROWB), off);
            }
            ec += BK;
            while (ec >= C) {
                ec -= C;
                if (++es == a.S) {
                    es = 0;
                    ++er;
                }
            }
        }
        {
            const uint32_t off = codes_valid ? (uint32_t)(((int64_t)fb * nchunks + chunk) * 1024 + lane * 16)
                                             : 0x80000000u;
            dma_b128(rs_c, st + L::B + (uint32_t)(cblk * 1024), off);
        }
        if constexpr (BWD) {
            // the stage's 32 bf16 scale pairs (every wave writes the same 128 bytes)
            const uint32_t off = lane < 32 ? (uint32_t)(chunk * 128 + lane * 4) : 0x80000000u;
            dma_b32(rs_p, st + L::P, off);
        }
    };

    // ---- operand addressing inside a stage ----
    const int sw = (l32 >> 1) & 7;  // row swizzle of this lane's MFMA rows
    int seg_off[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) seg_off[u] = 16 * ((2 * u + half) ^ sw);
    const int arow = (wm * WM + l32) * ROWB;
    const int bcol = (wn * WN + l32) * 16;
    uint32_t mk[4], shl[4];
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
        mk[jj] = 0x01010101u << (4 * half + jj);
        shl[jj] = 7 - 4 * half - jj;
    }

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int t = 0; t < TN; ++t)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][t][v] = 0.0f;

    // prologue: the first STAGES-1 stages in flight
#pragma unroll
    for (int c = 0; c < STAGES - 1; ++c)
        if (c < nloc) issue(c_begin + c);
    int cslot = 0;  // ring slot of the stage being multiplied
    for (int il = 0; il < niter; ++il) {
        // this wave's DMAs of stage il landed (later stages may still be in flight; in the
        // last stages simply everything)
        if (il + STAGES - 2 < nloc)
            wait_vmcnt((STAGES - 2) * DMAS);
        else
            wait_vmcnt(0);
        __syncthreads();  // ... and every other wave's; all reads of stage il-1 are done
        if (il + STAGES - 1 < nloc) issue(c_begin + il + STAGES - 1);  // into stage il-1's buffer
        if (G > 1 && il >= nloc) continue;  // past this group's range (wave-uniform)
        const uint8_t* st = ring + cslot * L::BYTES;
        cslot = cslot + 1 == STAGES ? 0 : cslot + 1;
        u32x4 braw[TN];
#pragma unroll
        for (int t = 0; t < TN; ++t) braw[t] = *reinterpret_cast<const u32x4*>(st + L::B + bcol + 32 * 16 * t);
        u32x4 base[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            if constexpr (BWD)
                base[u] = *reinterpret_cast<const u32x4*>(st + L::P + 32 * u + 16 * half);
            else
                base[u] = u32x4{0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u};
        }
        auto decode_b = [&](int u, bf16x8* bfr) {
#pragma unroll
            for (int t = 0; t < TN; ++t) {
                const uint32_t w = braw[t][u];
                u32x4 d;
                d.x = ((w & mk[0]) << shl[0]) + base[u].x;
                d.y = ((w & mk[1]) << shl[1]) + base[u].y;
                d.z = ((w & mk[2]) << shl[2]) + base[u].z;
                d.w = ((w & mk[3]) << shl[3]) + base[u].w;
                bfr[t] = as_bf16x8(d);
            }
        };
        auto read_a = [&](int u, bf16x8* af) {
#pragma unroll
            for (int i = 0; i < TM; ++i)
                af[i] = *reinterpret_cast<const bf16x8*>(st + L::A + arow + 32 * i * ROWB + seg_off[u]);
        };
        if constexpr (TM <= 4 && TM * TN < 8) {
            // small wave tiles: all of the stage's A operands are read up front so that
            // LDS latency overlaps the decode and the first MFMAs
            bf16x8 afs[4][TM];
#pragma unroll
            for (int u = 0; u < 4; ++u) read_a(u, afs[u]);
            __builtin_amdgcn_sched_barrier(0);  // keep the LDS reads ahead of the MFMAs
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                bf16x8 bfr[TN];
                decode_b(u, bfr);
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int t = 0; t < TN; ++t) acc[i][t] = mfma32(bfr[t], afs[u][i], acc[i][t]);
            }
        } else if constexpr (TM <= 4) {
            // 8 or more MFMAs per step: the A operands of step u + 1 are read and its filter
            // operand decoded while the MFMAs of step u run (one LDS read and two decode ops
            // after each MFMA); measured ~3-4% faster in the backward-data pass and ~1-2% in
            // the forward pass of the training layer than reading and decoding each step
            // right before its MFMAs
            bf16x8 afs[4][TM];
            bf16x8 bfr[2][TN];
            read_a(0, afs[0]);
            decode_b(0, bfr[0]);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                if (u + 1 < 4) {
                    read_a(u + 1, afs[u + 1]);
                    decode_b(u + 1, bfr[(u + 1) & 1]);
                }
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int t = 0; t < TN; ++t) acc[i][t] = mfma32(bfr[u & 1][t], afs[u][i], acc[i][t]);
                if (u + 1 < 4) {
#pragma unroll
                    for (int k = 0; k < TM; ++k) {
                        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
                        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
                        __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);  // two decode ops
                    }
#pragma unroll
                    for (int k = TM; k < TM * TN; ++k) {
                        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                        __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);
                    }
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        } else {
            // tall wave tiles: A operands one 16-element step ahead
            bf16x8 afc[TM], afn[TM];
            read_a(0, afc);
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                if (u < 3) read_a(u + 1, afn);
                bf16x8 bfr[TN];
                decode_b(u, bfr);
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int t = 0; t < TN; ++t) acc[i][t] = mfma32(bfr[t], afc[i], acc[i][t]);
                if (u < 3) {
#pragma unroll
                    for (int i = 0; i < TM; ++i) afc[i] = afn[i];
                }
            }
        }
    }

    // ---- epilogue.  The MFMA computed the transposed tile (filters x pixels): lane l of
    //      32x32 tile (i, t) holds pixel 32 i + l % 32 and, for each v / 4, four
    //      consecutive filters 32 t + 8 (v / 4) + 4 (l / 32) + 0..3.  Each 32-pixel tile row
    //      is staged through LDS with one 16-byte write per four filters, then every lane
    //      takes 8 consecutive channels of one pixel, applies y = act(acc * colscale *
    //      scale + bias + residual) and writes them with 16-byte stores. ----
    __syncthreads();  // every wave is done reading the ring
    if constexpr (G > 1) {
        // groups 1 .. G-1 store their sums (lane-contiguous 16-byte pieces), group 0 adds
        // them in group order
        f32x4* xch = reinterpret_cast<f32x4*>(smem + XOFF);
        if (grp > 0) {
            f32x4* dst = xch + (grp - 1) * (NACC / 4) * 256;
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int t = 0; t < TN; ++t)
#pragma unroll
                    for (int g4 = 0; g4 < 4; ++g4)
                        dst[(((i * TN + t) * 4 + g4) * 4 + wave) * 64 + lane] =
                            f32x4{acc[i][t][4 * g4], acc[i][t][4 * g4 + 1], acc[i][t][4 * g4 + 2], acc[i][t][4 * g4 + 3]};
        }
        __syncthreads();
        if (grp > 0) return;  // no barrier follows
#pragma unroll 1
        for (int gg = 1; gg < G; ++gg) {
            const f32x4* src = xch + (gg - 1) * (NACC / 4) * 256;
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int t = 0; t < TN; ++t)
#pragma unroll
                    for (int g4 = 0; g4 < 4; ++g4) {
                        const f32x4 v = src[(((i * TN + t) * 4 + g4) * 4 + wave) * 64 + lane];
                        acc[i][t][4 * g4] += v.x;
                        acc[i][t][4 * g4 + 1] += v.y;
                        acc[i][t][4 * g4 + 2] += v.z;
                        acc[i][t][4 * g4 + 3] += v.w;
                    }
        }
    }
    constexpr int PITCH = WN + 4;  // floats per staged pixel row
    float* stage = reinterpret_cast<float*>(smem) + wave * 32 * PITCH;
    const int Kf = a.Kf;
    constexpr int CG = WN / 8;    // 8-channel groups per pixel row of the wave tile
    constexpr int RPP = 64 / CG;  // pixel rows per pass
    const int gcol = lane % CG;
    const int grow = lane / CG;
    const int col0 = n0 + wn * WN + 8 * gcol;
    // bf16 residual: the 16-byte loads of PRE_I tile rows (at most 8 per lane) are issued
    // together before those rows are processed, so that their memory latency is paid once
    // per group rather than once per pass
    constexpr int NPASS = 32 / RPP;
    constexpr int PRE_I = NPASS >= 8 ? 1 : (8 / NPASS < TM ? 8 / NPASS : TM);
    static_assert(TM % PRE_I == 0, "residual prefetch groups");
    const uint16_t* res16 = reinterpret_cast<const uint16_t*>(a.residual);

    // Common case, decided per wave: bf16 output, no reduction split, the wave's tile wholly
    // inside the output (rows below M, whole 8-column groups below Kf) and 16-byte aligned
    // column factors.  It needs no per-row or per-column test: the column factors come in
    // with 16-byte loads and every pass is the same straight-line code.
    const bool fast = a.splits <= 1 && !a.y_f32 && (Kf % 8) == 0 && n0 + wn * WN + WN <= Kf &&
                      m0 + wm * WM + WM <= M &&
                      (((uintptr_t)a.colscale | (uintptr_t)a.scale | (uintptr_t)a.bias) & 15) == 0;
    if (fast) {
        f32x4 csl = {1.0f, 1.0f, 1.0f, 1.0f}, csh = csl, bil = {0.0f, 0.0f, 0.0f, 0.0f}, bih = bil;
        if (a.colscale) {
            csl = *reinterpret_cast<const f32x4*>(a.colscale + col0);
            csh = *reinterpret_cast<const f32x4*>(a.colscale + col0 + 4);
        }
        if (a.scale) {
            csl *= *reinterpret_cast<const f32x4*>(a.scale + col0);
            csh *= *reinterpret_cast<const f32x4*>(a.scale + col0 + 4);
        }
        if (a.bias) {
            bil = *reinterpret_cast<const f32x4*>(a.bias + col0);
            bih = *reinterpret_cast<const f32x4*>(a.bias + col0 + 4);
        }
        const float cs8[8] = {csl.x, csl.y, csl.z, csl.w, csh.x, csh.y, csh.z, csh.w};
        const float bi8[8] = {bil.x, bil.y, bil.z, bil.w, bih.x, bih.y, bih.z, bih.w};
        const bool res = a.residual != nullptr, relu = a.relu != 0;
        uint16_t* const y16 = reinterpret_cast<uint16_t*>(a.y);
        const int64_t rowb = m0 + wm * WM + grow;  // tile row 0 of this lane's passes
#pragma unroll
        for (int i0 = 0; i0 < TM; i0 += PRE_I) {
            u32x4 rpre[PRE_I][NPASS];
#pragma unroll
            for (int ii = 0; ii < PRE_I; ++ii)
#pragma unroll
                for (int pass = 0; pass < NPASS; ++pass)
                    rpre[ii][pass] = res ? *reinterpret_cast<const u32x4*>(res16 + (rowb + 32 * (i0 + ii) + pass * RPP) * Kf + col0)
                                         : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
            for (int ii = 0; ii < PRE_I; ++ii) {
                const int i = i0 + ii;
#pragma unroll
                for (int t = 0; t < TN; ++t)
#pragma unroll
                    for (int g = 0; g < 4; ++g)
                        *reinterpret_cast<f32x4*>(&stage[l32 * PITCH + 32 * t + 8 * g + 4 * half]) =
                            f32x4{acc[i][t][4 * g], acc[i][t][4 * g + 1], acc[i][t][4 * g + 2], acc[i][t][4 * g + 3]};
                __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this wave's LDS writes are visible to it
#pragma unroll
                for (int pass = 0; pass < NPASS; ++pass) {
                    const int r = pass * RPP + grow;
                    const f32x4 lo = *reinterpret_cast<const f32x4*>(&stage[r * PITCH + 8 * gcol]);
                    const f32x4 hi = *reinterpret_cast<const f32x4*>(&stage[r * PITCH + 8 * gcol + 4]);
                    float v8[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
#pragma unroll
                    for (int e = 0; e < 8; ++e) v8[e] = v8[e] * cs8[e] + bi8[e];
                    if (res) {
                        const u32x4 r8 = rpre[ii][pass];
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            v8[2 * e] += bf16_bits_to_f32(r8[e] & 0xFFFFu);
                            v8[2 * e + 1] += __uint_as_float(r8[e] & 0xFFFF0000u);
                        }
                    }
                    if (relu) {
#pragma unroll
                        for (int e = 0; e < 8; ++e) v8[e] = fmaxf(v8[e], 0.0f);
                    }
                    const u32x4 out = u32x4{pack_bf16x2(v8[0], v8[1]), pack_bf16x2(v8[2], v8[3]),
                                            pack_bf16x2(v8[4], v8[5]), pack_bf16x2(v8[6], v8[7])};
                    u32x4* const dst = reinterpret_cast<u32x4*>(y16 + (rowb + 32 * i + pass * RPP) * Kf + col0);
                    if (a.y_stream)
                        __builtin_nontemporal_store(out, dst);
                    else
                        *dst = out;
                }
                __builtin_amdgcn_s_waitcnt(0xC07F);  // reads of this tile row done before it is overwritten
            }
        }
        return;
    }

    float cs[8], bi[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const int col = col0 + e;
        const bool ok = col < Kf;
        float sc = ok && a.colscale ? a.colscale[col] : 1.0f;
        if (ok && a.scale) sc *= a.scale[col];
        cs[e] = sc;
        bi[e] = ok && a.bias ? a.bias[col] : 0.0f;
    }
    const bool vec_store = (Kf % 8) == 0;
    const bool partial_out = a.splits > 1;  // raw fp32 sums of this split, rows of Kp = round_up(Kf, 8)
    const int Kp = (Kf + 7) & ~7;
    float* part = partial_out ? a.partial + (int64_t)split * M * Kp : nullptr;
    const bool res_pre = a.residual && !a.y_f32 && vec_store && !partial_out && col0 < Kf;
#pragma unroll
    for (int i0 = 0; i0 < TM; i0 += PRE_I) {
        u32x4 rpre[PRE_I][NPASS];
#pragma unroll
        for (int ii = 0; ii < PRE_I; ++ii)
#pragma unroll
            for (int pass = 0; pass < NPASS; ++pass) {
                const int64_t row = m0 + wm * WM + 32 * (i0 + ii) + pass * RPP + grow;
                rpre[ii][pass] = res_pre && row < M ? *reinterpret_cast<const u32x4*>(res16 + row * Kf + col0)
                                                    : u32x4{0u, 0u, 0u, 0u};
            }
#pragma unroll
        for (int ii = 0; ii < PRE_I; ++ii) {
            const int i = i0 + ii;
#pragma unroll
            for (int t = 0; t < TN; ++t)
#pragma unroll
                for (int g = 0; g < 4; ++g)
                    *reinterpret_cast<f32x4*>(&stage[l32 * PITCH + 32 * t + 8 * g + 4 * half]) =
                        f32x4{acc[i][t][4 * g], acc[i][t][4 * g + 1], acc[i][t][4 * g + 2], acc[i][t][4 * g + 3]};
            __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this wave's LDS writes are visible to it
#pragma unroll
            for (int pass = 0; pass < 32 / RPP; ++pass) {
                const int r = pass * RPP + grow;
                const int64_t row = m0 + wm * WM + 32 * i + r;
                if (row >= M) continue;
                const f32x4 lo = *reinterpret_cast<const f32x4*>(&stage[r * PITCH + 8 * gcol]);
                const f32x4 hi = *reinterpret_cast<const f32x4*>(&stage[r * PITCH + 8 * gcol + 4]);
                float v8[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
                const int64_t o = row * Kf + col0;
                if (partial_out) {
                    if (col0 < Kf) {
                        float* pp = part + row * Kp + col0;
                        *reinterpret_cast<f32x4*>(pp) = lo;
                        *reinterpret_cast<f32x4*>(pp + 4) = hi;
                    }
                    continue;
                }
#pragma unroll
                for (int e = 0; e < 8; ++e) v8[e] = v8[e] * cs[e] + bi[e];
                if (a.residual) {
                    if (a.y_f32) {
                        const float* rp = reinterpret_cast<const float*>(a.residual) + o;
#pragma unroll
                        for (int e = 0; e < 8; ++e)
                            if (col0 + e < Kf) v8[e] += rp[e];
                    } else {
                        const uint16_t* rp = reinterpret_cast<const uint16_t*>(a.residual) + o;
                        if (vec_store && col0 < Kf) {
                            const u32x4 r8 = rpre[ii][pass];
#pragma unroll
                            for (int e = 0; e < 4; ++e) {
                                v8[2 * e] += bf16_bits_to_f32(r8[e] & 0xFFFFu);
                                v8[2 * e + 1] += bf16_bits_to_f32(r8[e] >> 16);
                            }
                        } else {
#pragma unroll
                            for (int e = 0; e < 8; ++e)
                                if (col0 + e < Kf) v8[e] += bf16_bits_to_f32(rp[e]);
                        }
                    }
                }
                if (a.relu) {
#pragma unroll
                    for (int e = 0; e < 8; ++e) v8[e] = fmaxf(v8[e], 0.0f);
                }
                if (a.y_f32) {
                    float* yp = reinterpret_cast<float*>(a.y) + o;
                    if (vec_store && col0 < Kf) {
                        *reinterpret_cast<f32x4*>(yp) = f32x4{v8[0], v8[1], v8[2], v8[3]};
                        *reinterpret_cast<f32x4*>(yp + 4) = f32x4{v8[4], v8[5], v8[6], v8[7]};
                    } else {
#pragma unroll
                        for (int e = 0; e < 8; ++e)
                            if (col0 + e < Kf) yp[e] = v8[e];
                    }
                } else {
                    uint16_t* yp = reinterpret_cast<uint16_t*>(a.y) + o;
                    if (vec_store && col0 < Kf) {
                        *reinterpret_cast<u32x4*>(yp) = u32x4{pack_bf16x2(v8[0], v8[1]), pack_bf16x2(v8[2], v8[3]),
                                                              pack_bf16x2(v8[4], v8[5]), pack_bf16x2(v8[6], v8[7])};
                    } else {
#pragma unroll
                        for (int e = 0; e < 8; ++e)
                            if (col0 + e < Kf) yp[e] = (uint16_t)f32_to_bf16_bits(v8[e]);
                    }
                }
            }
            __builtin_amdgcn_s_waitcnt(0xC07F);  // reads of this tile row done before it is overwritten
        }
    }
}

// Sum of the split-K partials in split order, then the epilogue; one thread per 8 outputs.
__global__ __launch_bounds__(256) void conv_split_epilogue_kernel(const ConvGemmArgs a) {
    const int64_t M = (int64_t)a.N * a.P * a.Q;
    const int Kp = (a.Kf + 7) & ~7;
    const int64_t groups = M * (Kp / 8);
    const int64_t gi = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (gi >= groups) return;
    const int64_t row = gi / (Kp / 8);
    split_epilogue_group(a, M, row, (int)(gi - row * (Kp / 8)) * 8);
}

template <int BM, int BN, int WAVES_M, int WAVES_N, int STAGES, bool BWD, int G = 1>
hipError_t launch_dma_cfg(const ConvGemmArgs& args, hipStream_t stream) {
    ConvGemmArgs a = args;
    const int64_t M = (int64_t)a.N * a.P * a.Q;
    const int64_t tilesN = (a.Kf + BN - 1) / BN;
    const int64_t tiles = ((M + BM - 1) / BM) * tilesN;
    if (tiles * a.splits >= 0x7FFFFFFFll) return hipErrorInvalidValue;
    a.div_tiles = make_fastdiv((uint32_t)tiles);
    a.div_tilesN = make_fastdiv((uint32_t)tilesN);
    uint64_t rep = 0;
    for (int r = 0; r < a.R; ++r) rep |= 1ull << (r * a.S);
    a.rep_lo = (uint32_t)rep;
    a.rep_hi = (uint32_t)(rep >> 32);
    const dim3 grid((unsigned)(tiles * a.splits));
    if (a.C % 64 == 0)
        hipLaunchKernelGGL((conv_dma_kernel<BM, BN, WAVES_M, WAVES_N, STAGES, BWD, true, G>), grid, dim3(256 * G), 0, stream, a);
    else
        hipLaunchKernelGGL((conv_dma_kernel<BM, BN, WAVES_M, WAVES_N, STAGES, BWD, false, G>), grid, dim3(256 * G), 0, stream, a);
    return hipGetLastError();
}

template <bool BWD>
hipError_t launch_dma_mode(const ConvGemmArgs& a, int cfg, hipStream_t stream) {
    switch (cfg) {
        case 11: return launch_dma_cfg<128, 128, 1, 4, 3, BWD>(a, stream);
        case 12: return launch_dma_cfg<128, 128, 2, 2, 3, BWD>(a, stream);
        case 13: return launch_dma_cfg<128, 128, 1, 4, 4, BWD>(a, stream);
        case 14: return launch_dma_cfg<128, 64, 2, 2, 3, BWD>(a, stream);
        case 16: return launch_dma_cfg<256, 128, 1, 4, 2, BWD>(a, stream);
        case 18: return launch_dma_cfg<64, 128, 1, 4, 4, BWD>(a, stream);
        case 19: return launch_dma_cfg<256, 256, 2, 2, 3, BWD>(a, stream);
        case 17: return launch_dma_cfg<256, 256, 2, 2, 4, BWD>(a, stream);
        case 21: return launch_dma_cfg<64, 128, 1, 4, 4, BWD, 2>(a, stream);
        case 22: return launch_dma_cfg<64, 128, 1, 4, 3, BWD, 4>(a, stream);
        case 23: return launch_dma_cfg<128, 128, 1, 4, 4, BWD, 2>(a, stream);
        case 24: return launch_dma_cfg<128, 64, 2, 2, 3, BWD, 2>(a, stream);
        case 25: return launch_dma_cfg<64, 128, 1, 4, 3, BWD, 2>(a, stream);
        default: return launch_dma_cfg<128, 256, 1, 4, 3, BWD>(a, stream);
    }
}

// groups of four waves per block (each reducing its own range of stages)
int cfg_groups(int cfg) { return cfg == 22 ? 4 : (cfg == 21 || cfg == 23 || cfg == 24 || cfg == 25) ? 2 : 1; }

void cfg_tile(int cfg, int* bm, int* bn) {
    switch (cfg) {
        case 11: case 12: case 13: *bm = 128; *bn = 128; return;
        case 14: *bm = 128; *bn = 64; return;
        case 18: case 21: case 22: case 25: *bm = 64; *bn = 128; return;
        case 23: *bm = 128; *bn = 128; return;
        case 24: *bm = 128; *bn = 64; return;
        case 16: *bm = 256; *bn = 128; return;
        case 17: case 19: *bm = 256; *bn = 256; return;
        default: *bm = 128; *bn = 256; return;
    }
}

}  // namespace

bool conv_dma_eligible(const ConvGemmArgs& a) {
    const int64_t xbytes = (int64_t)a.N * a.H * a.W * a.C * 2;
    const int64_t nchunks = ((int64_t)a.R * a.S * a.C + BK - 1) / BK;
    const int64_t cbytes = (int64_t)((a.Kf + 63) / 64) * nchunks * 1024;
    return !a.x_f32 && a.C % 8 == 0 && a.R * a.S <= 63 && xbytes < 0x7FFFFFF0ll && cbytes < 0x7FFFFFF0ll;
}

ConvPlan plan_conv_dma(const ConvGemmArgs& a, int cfg) {
    const int64_t M = (int64_t)a.N * a.P * a.Q;
    const int nchunks = (int)(((int64_t)a.R * a.S * a.C + BK - 1) / BK);
    ConvPlan p;
    p.cfg = cfg;
    int bm, bn;
    if (p.cfg < 10) {
        // 65..128 filters: 128 x 128 tiles with one wave per 32 filters (each wave decodes
        // only its own filters), measured ~4-8% faster than two waves per 64 filters on the
        // ResNet-18 layer-2 shapes, and a three-deep ring (there 4-8% faster than four deep)
        p.cfg = a.Kf > 128 ? 10 : (a.Kf > 64 ? 11 : 14);
        cfg_tile(p.cfg, &bm, &bn);
        // too few tiles for one wave of blocks: shorter tiles (64 pixels x 128 filters, a
        // four-deep ring) when there are at least 128 filters, else 128 x 64; then split
        // the reduction
        if (((M + bm - 1) / bm) * ((a.Kf + bn - 1) / bn) < 384) p.cfg = a.Kf >= 128 ? 18 : 14;
        // 128 .. 255 tiles of 64 x 128: one block per CU, so four groups of four waves per
        // block (four waves per SIMD) instead of a reduction split; measured 23 vs 31-34 us
        // on the 7 x 7 x 512 ResNet-18 layers at batch 64
        if (p.cfg == 18) {
            const int64_t t18 = ((M + 63) / 64) * ((a.Kf + 127) / 128);
            if (t18 >= 128 && t18 < 256 && nchunks >= 16) p.cfg = 22;
            // fewer than 128 tiles (batch-1 layers): two or four wave groups per block
            // splitting the reduction inside the block, instead of a grid split and its
            // epilogue pass, when every group then has 4 to 10 stages.  Measured on the
            // ResNet-18 batch-1 layers: 28 x 28 x 128, two groups of 9 stages, 9.0 us against
            // 12.3 us split three ways plus the epilogue pass; 14 x 14 x 256, four groups of
            // 9, 12.7 against 13.0 us; 7 x 7 x 512 (18 stages per group with four groups)
            // stays split: 13.4 against 20.8 us.
            if (t18 < 128) {
                if (nchunks >= 8 && (nchunks + 1) / 2 <= 10)
                    p.cfg = 21;
                else if (nchunks >= 16 && (nchunks + 3) / 4 <= 10)
                    p.cfg = 22;
            }
        }
    }
    cfg_tile(p.cfg, &bm, &bn);
    const int64_t tiles = ((M + bm - 1) / bm) * ((a.Kf + bn - 1) / bn);
    int64_t splits = 1;
    {
        const int forced = conv_splits_override();
        if (forced > 0) {
            splits = forced;
        } else if (tiles < 384 && cfg_groups(p.cfg) == 1) {
            // measured: the 64 x 128 tile split only below ~192 tiles (then to about 192
            // blocks with >= 6 stages each: a split costs a partial-sum pass), the 128 x 64
            // tile to about 640 blocks with >= 6 stages each (the 3 x 3 x 64 layer at batch 1,
            // 9 stages, runs 8.8 us unsplit against 10.8 us in three ranges)
            const bool shortt = p.cfg == 18;
            const int64_t target = shortt ? 192 : 640, min_stages = 6;
            splits = (target + tiles - 1) / tiles;
            const int64_t max_splits = nchunks / min_stages > 0 ? nchunks / min_stages : 1;
            if (splits > max_splits) splits = max_splits;
        }
        if (splits > nchunks) splits = nchunks;
        if (splits < 1) splits = 1;
    }
    // each block's G groups take G consecutive ranges of chunks_per_split stages
    const int G = cfg_groups(p.cfg);
    p.chunks_per_split = (int)((nchunks + splits * G - 1) / (splits * G));
    p.splits = (int)((nchunks + (int64_t)p.chunks_per_split * G - 1) / ((int64_t)p.chunks_per_split * G));
    // partial rows padded to whole 8-column groups
    p.partial_bytes = p.splits > 1 ? (size_t)p.splits * (size_t)M * (size_t)((a.Kf + 7) & ~7) * 4 : 0;
    return p;
}

hipError_t launch_conv_dma(const ConvGemmArgs& args, const ConvPlan& plan, hipStream_t stream) {
    ConvGemmArgs a = args;
    a.splits = plan.splits;
    a.chunks_per_split = plan.chunks_per_split;
    if (a.splits > 1 && !a.partial) return hipErrorInvalidValue;
    // outputs of 128 MiB and more (half the 256 MB last-level cache) are written with
    // streaming stores: the next layer reads most of them from HBM in any case, and keeping
    // them out of the caches measured 2-4% faster on the 128 x 56 x 56 x 256 layer, while
    // smaller outputs (every ResNet-18 layer at batch 64) stay cached for the next layer
    a.y_stream = (int64_t)a.N * a.P * a.Q * a.Kf * (a.y_f32 ? 4 : 2) >= (128ll << 20) ? 1 : 0;
    hipError_t e = a.apair ? launch_dma_mode<true>(a, plan.cfg, stream) : launch_dma_mode<false>(a, plan.cfg, stream);
    if (e != hipSuccess || a.splits <= 1) return e;
    const int64_t groups = (int64_t)a.N * a.P * a.Q * (((a.Kf + 7) & ~7) / 8);
    hipLaunchKernelGGL(conv_split_epilogue_kernel, dim3((unsigned)((groups + 255) / 256)), dim3(256), 0, stream, a);
    return hipGetLastError();
}

}  // namespace tbn
