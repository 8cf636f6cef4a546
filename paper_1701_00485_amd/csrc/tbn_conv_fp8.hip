// tbn_conv_fp8.hip -- forward pass of a two-bit layer on fp8 activation codes: Eq. (1) with
// the input replaced by s * f (f an E4M3 value, one fp32 scale s per tensor), on the gfx950
// scaled matrix cores (v_mfma_scale_f32_32x32x64_f8f6f4 with unit scales): the filter values
// +-1 and +-2 are exact in the 4-bit E2M1 format, every product f * W~ is exact and the sums
// are fp32.  Also the E4M3 activation codes and the repack of the packed filter codes into
// the E2M1 operand layout.
//
// The convolution follows the int8 kernel (implicit GEMM; activation rows and code blocks
// copied to LDS by buffer loads in LDS-DMA mode, a three-deep ring with compile-time vmcnt
// waits, swizzled 128-byte rows, XCD-aware tile order), with stages of 128 channels (one
// byte each) and two MFMA steps of 64 reduction elements, one 64-element code chunk each.
//   * Operand layout of the MFMA (measured): an E2M1 operand lane of lane-half h holds
//     reduction elements 32 h .. 32 h + 31 of the step in its 32 nibbles; an E4M3 operand
//     lane of lane-half h holds elements 16 h .. 16 h + 15 in bytes 0-15 and 32 + 16 h ..
//     32 + 16 h + 15 in bytes 16-31.  So a lane's activation operand of step t is two
//     16-byte segments of the row (4 t + h and 4 t + 2 + h), and its filter operand the
//     words 2 h and 2 h + 1 of the filter's code chunk t.
//   * The filters are read in the E2M1 layout made by the repack kernel: the same 16 bytes
//     per filter and 64-element chunk as the packed codes, but word q holds elements
//     16 q + 8 r + j (r = 0, 1; j = 0..7) as magnitude bit 4 j + 1 - r and sign bit
//     4 j + 3 - r, so that 8 E2M1 values (2 + 2 magnitude + 8 sign per nibble: 1.0, 2.0,
//     -1.0, -2.0) are one mask and one add (r = 0) or a mask and a shift-add (r = 1).
//   * The epilogue multiplies the fp32 sums by fp32(alpha_k * s), optionally clamps at 0 and
//     stores bf16 or fp32 through an LDS staging tile with 16-byte stores.
//
// M0 is written by the DMA helper; nothing else in these kernels uses M0.
#include "tbn_device.h"
#include "tbn_dma.h"
#include "tbn_kernels.h"

namespace tbn {

namespace {

constexpr int BK = 128;    // fp8 reduction elements per stage
constexpr int ROWB = 128;  // LDS bytes per activation row of a stage

template <int BM, int BN>
struct Fp8Layout {
    static constexpr int A = 0;            // BM rows x 128 B
    static constexpr int B = BM * ROWB;    // code chunk 0 of the BN filters, then chunk 1
    static constexpr int BYTES = B + 2 * BN * 16;
};

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x8 __attribute__((ext_vector_type(8)));

// D += A B with A the E2M1 filter operand (format 4) and B the E4M3 activation operand
// (format 0), both scales 2^0 (E8M0 code 127)
__device__ __forceinline__ f32x16 mfma_f4f8(i32x8 fil, i32x8 act, f32x16 c) {
    return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(fil, act, c, 4, 0, 0, 127, 0, 127);
}

// (t << 1) + c in one v_lshl_add_u32 (c in a scalar register: the three-operand form takes
// no literal)
__device__ __forceinline__ uint32_t shl1_add(uint32_t t, uint32_t c) {
    uint32_t r;
    asm("v_lshl_add_u32 %0, %1, 1, %2" : "=v"(r) : "v"(t), "s"(c));
    return r;
}

// The 32 E2M1 values of words w0 (elements 0..15) and w1 (16..31) of the repacked layout;
// two22 = 0x22222222 (the 2 of every nibble) in a scalar register.
__device__ __forceinline__ i32x8 decode_f4(uint32_t w0, uint32_t w1, uint32_t two22) {
    i32x4 r;
    r[0] = (int)((w0 & 0xAAAAAAAAu) + two22);
    r[1] = (int)shl1_add(w0 & 0x55555555u, two22);
    r[2] = (int)((w1 & 0xAAAAAAAAu) + two22);
    r[3] = (int)shl1_add(w1 & 0x55555555u, two22);
    // the E2M1 form reads only the low four dwords: the others are left undefined
    return __builtin_shufflevector(r, r, 0, 1, 2, 3, -1, -1, -1, -1);
}

// UNI: C % 128 == 0, so all 128 elements of a stage share one tap (r, s) and the tap
// bookkeeping is wave-uniform.  Otherwise C % 16 == 0 and every lane tracks the tap of its
// own 16-channel segment.
template <int BM, int BN, int WAVES_M, int WAVES_N, int STAGES, bool UNI>
__global__ __launch_bounds__(256, 2) void conv_fp8_kernel(const ConvFp8Args a) {
    constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
    constexpr int TM = WM / 32, TN = WN / 32;
    constexpr int AR = BM / 32;    // activation DMAs per wave per stage (8 rows each)
    constexpr int NBLK = BN / 64;  // 1 KiB code blocks per chunk
    using L = Fp8Layout<BM, BN>;
    static_assert(WAVES_M * WAVES_N == 4, "four waves per block");
    static_assert(TM >= 1 && TN >= 1 && BM % 32 == 0 && BN % 64 == 0 && NBLK <= 4, "tile shape");
    static_assert(STAGES * L::BYTES >= 4 * 32 * (WN + 4) * 4, "epilogue staging fits in the ring");

    __shared__ __attribute__((aligned(1024))) uint8_t smem[STAGES * L::BYTES];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / WAVES_N;
    const int wn = wave % WAVES_N;
    const int half = lane >> 5;
    const int l32 = lane & 31;

    const int64_t PQ = (int64_t)a.P * a.Q;
    const int64_t M = (int64_t)a.N * PQ;
    const int C = a.C;
    const int n = a.R * a.S * C;
    const int nst = (n + BK - 1) / BK;  // stages
    const int nch = (n + 63) / 64;      // 64-element code chunks
    const int KB = (a.K + 63) / 64;
    const uint32_t tilesN = (uint32_t)(a.K + BN - 1) / BN;
    const uint32_t tile = (uint32_t)xcd_remap(blockIdx.x, gridDim.x);
    const uint32_t mtile = fdiv(tile, a.div_tilesN);
    const int64_t m0 = (int64_t)mtile * BM;
    const int n0 = (int)(tile - mtile * tilesN) * BN;

    const v4i rs_x = make_rsrc(a.x, (uint32_t)((int64_t)a.N * a.H * a.W * C));
    const v4i rs_c = make_rsrc(a.codes, (uint32_t)((int64_t)KB * nch * 1024));
    const uint32_t smem_base = lds_addr(smem);

    // ---- activation rows this lane fills: row = 8 * (wave + 4 j) + lane / 8 ----
    int32_t rbase[AR];      // byte offset of the row's (h0, w0) in x (may be negative)
    uint32_t rmask[AR][2];  // bit r*S + s set iff tap (r, s) lies inside the image
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
            // in-image taps s in [slo, shi), r in [rlo, rhi): the row's bits replicated at
            // every in-image r by a multiplication with sum_r 2^(r*S) (R*S <= 63)
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
    // logical 16-byte segment this lane loads (its LDS slot is lane % 8 of the row; rows
    // swizzled by (row / 2) % 8)
    const int lseg = (lane & 7) ^ ((4 * (wave & 1)) | ((lane >> 4) & 3));
    int er = 0, es = 0, ec = 0;  // general path: (r, s, c) of this lane's next segment
    int us = 0, uc = 0, utap = 0;  // uniform path: s, first channel and tap of the next stage
    uint32_t utoff = 0;            // uniform path: byte offset of (r, s, c0) from a row's (h0, w0)
    uint32_t rbs[AR];              // uniform path: row offset plus this lane's segment
    uint32_t nmask[AR][2];         // uniform path: complement of rmask
    if constexpr (UNI) {
#pragma unroll
        for (int j = 0; j < AR; ++j) {
            rbs[j] = (uint32_t)(rbase[j] + 16 * lseg);
            nmask[j][0] = ~rmask[j][0];
            nmask[j][1] = ~rmask[j][1];
        }
    } else {
        const int e0 = lseg * 16;
        const int rs = e0 / C;
        ec = e0 - rs * C;
        er = rs / a.S;
        es = rs - er * a.S;
    }
    // code blocks of this wave: block wave % NBLK of both chunks of each stage (with fewer
    // than four blocks some waves copy identical bytes to the same place), so that every
    // wave issues the same number of DMAs per stage and the waits are compile-time counts
    const int cblk = wave % NBLK;
    const int fb = n0 / 64 + cblk;
    const bool codes_valid = fb < KB;
    constexpr int DMAS = AR + 2;

    const uint32_t row_step = (uint32_t)((a.W - a.S) * C);  // to the next filter row, bytes
    int islot = 0;
    auto issue = [&](int stage) {
        const uint32_t st = smem_base + (uint32_t)(islot * L::BYTES);
        islot = islot + 1 == STAGES ? 0 : islot + 1;
        if constexpr (UNI) {
            // out-of-image taps and the taps past the filter (clamped to bit 63, clear
            // because R*S <= 63) get offset bit 31 set: the hardware returns zeros
            const int tap = min(utap, 63);
            if (tap < 32) {
#pragma unroll
                for (int j = 0; j < AR; ++j) {
                    const uint32_t out = (nmask[j][0] << (31 - tap)) & 0x80000000u;
                    dma_b128(rs_x, st + L::A + (uint32_t)(8 * (wave + 4 * j) * ROWB), (rbs[j] + utoff) | out);
                }
            } else {
#pragma unroll
                for (int j = 0; j < AR; ++j) {
                    const uint32_t out = (nmask[j][1] << (63 - tap)) & 0x80000000u;
                    dma_b128(rs_x, st + L::A + (uint32_t)(8 * (wave + 4 * j) * ROWB), (rbs[j] + utoff) | out);
                }
            }
            uc += BK;
            utoff += BK;
            if (uc == C) {
                uc = 0;
                ++utap;
                if (++us == a.S) {
                    us = 0;
                    utoff += row_step;
                }
            }
        } else {
            const int tap = min(er * a.S + es, 63);
            const int tword = tap >> 5, tbit = tap & 31;
            const int32_t toff = (er * a.W + es) * C + ec;
#pragma unroll
            for (int j = 0; j < AR; ++j) {
                const bool ok = ((tword ? rmask[j][1] : rmask[j][0]) >> tbit) & 1u;
                const uint32_t off = ok ? (uint32_t)(rbase[j] + toff) : 0x80000000u;
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
#pragma unroll
        for (int cc = 0; cc < 2; ++cc) {
            const int ch = 2 * stage + cc;
            const uint32_t off = (codes_valid && ch < nch) ? (uint32_t)(((int64_t)fb * nch + ch) * 1024 + lane * 16)
                                                           : 0x80000000u;
            dma_b128(rs_c, st + L::B + (uint32_t)((cc * NBLK + cblk) * 1024), off);
        }
    };

    // ---- operand addressing inside a stage ----
    const int sw = (l32 >> 1) & 7;
    // the two 16-byte activation segments of step t: logical 4 t + half and 4 t + 2 + half
    int seg_lo[2], seg_hi[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
        seg_lo[t] = 16 * ((4 * t + half) ^ sw);
        seg_hi[t] = 16 * ((4 * t + 2 + half) ^ sw);
    }
    const int arow = (wm * WM + l32) * ROWB;
    const int bcol = (wn * WN + l32) * 16 + 8 * half;  // words 2 half, 2 half + 1 of a chunk row
    const uint32_t two22 = __builtin_amdgcn_readfirstlane(0x22222222u);

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int t = 0; t < TN; ++t)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][t][v] = 0.0f;

#pragma unroll
    for (int c = 0; c < STAGES - 1; ++c)
        if (c < nst) issue(c);
    int cslot = 0;
    for (int il = 0; il < nst; ++il) {
        if (il + STAGES - 2 < nst)
            wait_vmcnt((STAGES - 2) * DMAS);
        else
            wait_vmcnt(0);
        __syncthreads();  // every wave's copies of stage il landed; reads of il-1 are done
        if (il + STAGES - 1 < nst) issue(il + STAGES - 1);
        const uint8_t* st = smem + cslot * L::BYTES;
        cslot = cslot + 1 == STAGES ? 0 : cslot + 1;
        // step 0's operands first; step 1's are read between step 0's MFMAs
        i32x8 af[2][TM];
        u32x2 bw[2][TN];
        auto read_step = [&](int s2) {
#pragma unroll
            for (int t = 0; t < TN; ++t)
                bw[s2][t] = *reinterpret_cast<const u32x2*>(st + L::B + s2 * NBLK * 1024 + bcol + 32 * 16 * t);
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                const uint8_t* rp = st + L::A + arow + 32 * i * ROWB;
                const i32x4 lo = *reinterpret_cast<const i32x4*>(rp + seg_lo[s2]);
                const i32x4 hi = *reinterpret_cast<const i32x4*>(rp + seg_hi[s2]);
                af[s2][i] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
            }
        };
        read_step(0);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
            if (s2 == 0) read_step(1);
#pragma unroll
            for (int t = 0; t < TN; ++t) {
                const i32x8 bf = decode_f4(bw[s2][t].x, bw[s2][t].y, two22);
#pragma unroll
                for (int i = 0; i < TM; ++i) acc[i][t] = mfma_f4f8(bf, af[s2][i], acc[i][t]);
            }
            if (s2 == 0) {
                // two LDS reads after each MFMA
#pragma unroll
                for (int k = 0; k < TM * TN; ++k) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
                    __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // two LDS reads
                }
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    }

    // ---- epilogue.  The MFMA computed the transposed tile (filters x pixels): lane l of
    //      tile (i, t) holds pixel 32 i + l % 32 and, for each v / 4, filters
    //      32 t + 8 (v / 4) + 4 (l / 32) + 0..3.  Each 32-pixel tile row is staged through
    //      LDS, then every lane scales 8 consecutive channels of one pixel. ----
    __syncthreads();
    constexpr int PITCH = WN + 4;
    float* stage = reinterpret_cast<float*>(smem) + wave * 32 * PITCH;
    const int K = a.K;
    constexpr int CG = WN / 8;
    constexpr int RPP = 64 / CG;
    const int gcol = lane % CG;
    const int grow = lane / CG;
    const int col0 = n0 + wn * WN + 8 * gcol;
    float cs[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) cs[e] = col0 + e < K ? a.alpha[col0 + e] * a.x_scale : 0.0f;
    const bool vec_store = (K % 8) == 0;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
        for (int t = 0; t < TN; ++t)
#pragma unroll
            for (int g = 0; g < 4; ++g)
                *reinterpret_cast<f32x4*>(&stage[l32 * PITCH + 32 * t + 8 * g + 4 * half]) =
                    f32x4{acc[i][t][4 * g], acc[i][t][4 * g + 1], acc[i][t][4 * g + 2], acc[i][t][4 * g + 3]};
        __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
#pragma unroll
        for (int pass = 0; pass < 32 / RPP; ++pass) {
            const int r = pass * RPP + grow;
            const int64_t row = m0 + wm * WM + 32 * i + r;
            if (row >= M || col0 >= K) continue;
            const f32x4 lo = *reinterpret_cast<const f32x4*>(&stage[r * PITCH + 8 * gcol]);
            const f32x4 hi = *reinterpret_cast<const f32x4*>(&stage[r * PITCH + 8 * gcol + 4]);
            float v8[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
#pragma unroll
            for (int e = 0; e < 8; ++e) v8[e] = v8[e] * cs[e];
            if (a.relu) {
#pragma unroll
                for (int e = 0; e < 8; ++e) v8[e] = fmaxf(v8[e], 0.0f);
            }
            const int64_t o = row * K + col0;
            if (a.y_f32) {
                float* yp = reinterpret_cast<float*>(a.y) + o;
                if (vec_store) {
                    *reinterpret_cast<f32x4*>(yp) = f32x4{v8[0], v8[1], v8[2], v8[3]};
                    *reinterpret_cast<f32x4*>(yp + 4) = f32x4{v8[4], v8[5], v8[6], v8[7]};
                } else {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if (col0 + e < K) yp[e] = v8[e];
                }
            } else {
                uint16_t* yp = reinterpret_cast<uint16_t*>(a.y) + o;
                if (vec_store) {
                    *reinterpret_cast<u32x4*>(yp) = u32x4{pack_bf16x2(v8[0], v8[1]), pack_bf16x2(v8[2], v8[3]),
                                                          pack_bf16x2(v8[4], v8[5]), pack_bf16x2(v8[6], v8[7])};
                } else {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if (col0 + e < K) yp[e] = (uint16_t)f32_to_bf16_bits(v8[e]);
                }
            }
        }
        __builtin_amdgcn_s_waitcnt(0xC07F);  // reads of this tile row done before it is overwritten
    }
}

// E4M3 code of one fp32 value: nearest, ties to even, |v| > 448 -> +-448, NaN -> 0, the
// sign bit kept for -0 and values that round to zero.  Below 2^-6 the codes are the
// subnormals, v / 2^-9 rounded to an integer 0..8 (8 is the smallest normal, 0x08); above,
// code = 8 (e + 7) + m with m = (v / 2^e - 1) * 8 rounded to an integer 0..8 (8 carries into
// the exponent field).  Every scaling here is by a power of two, so exact, and rintf rounds
// half to even.
__device__ __forceinline__ uint32_t fp8_code(float v) {
    const uint32_t bits = __float_as_uint(v);
    const uint32_t sign = (bits >> 24) & 0x80u;
    const float av = fabsf(v);
    uint32_t mag;
    if (!(av <= 448.0f)) {
        mag = av != av ? 0xFFFFFFFFu : 0x7Eu;  // NaN marked, overflow saturates
    } else if (av < 0.015625f) {
        mag = (uint32_t)rintf(av * 512.0f);
    } else {
        const int e = (int)((__float_as_uint(av) >> 23) & 0xFF) - 127;  // av normal in fp32 here
        const float frac = __uint_as_float((__float_as_uint(av) & 0x007FFFFFu) | 0x3F800000u);  // av / 2^e
        mag = (uint32_t)(8 * (e + 7)) + (uint32_t)rintf((frac - 1.0f) * 8.0f);
    }
    return mag == 0xFFFFFFFFu ? 0u : (sign | mag);
}

// codes of 16 activations per thread (v = x * inv in fp32 first)
template <bool F32>
__global__ __launch_bounds__(256) void quantize_act_fp8_kernel(const void* __restrict__ x, int64_t count, float inv,
                                                               uint8_t* __restrict__ q) {
    const int64_t i0 = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 16;
    if (i0 >= count) return;
    float v[16];
    const bool full = i0 + 16 <= count;
    if (full) {
        if constexpr (F32) {
            const f32x4* p = reinterpret_cast<const f32x4*>(reinterpret_cast<const float*>(x) + i0);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const f32x4 t = p[j];
                v[4 * j] = t.x; v[4 * j + 1] = t.y; v[4 * j + 2] = t.z; v[4 * j + 3] = t.w;
            }
        } else {
            const u32x4* p = reinterpret_cast<const u32x4*>(reinterpret_cast<const uint16_t*>(x) + i0);
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const u32x4 t = p[j];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    v[8 * j + 2 * e] = bf16_bits_to_f32(t[e] & 0xFFFFu);
                    v[8 * j + 2 * e + 1] = bf16_bits_to_f32(t[e] >> 16);
                }
            }
        }
    } else {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const int64_t i = i0 + e < count ? i0 + e : i0;
            v[e] = F32 ? reinterpret_cast<const float*>(x)[i] : bf16_bits_to_f32(reinterpret_cast<const uint16_t*>(x)[i]);
        }
    }
    uint32_t word[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int e = 0; e < 16; ++e) word[e / 4] |= fp8_code(v[e] * inv) << (8 * (e % 4));
    if (full) {
        *reinterpret_cast<u32x4*>(q + i0) = u32x4{word[0], word[1], word[2], word[3]};
    } else {
        for (int e = 0; i0 + e < count; ++e) q[i0 + e] = (uint8_t)((word[e / 4] >> (8 * (e % 4))) & 0xFFu);
    }
}

// One packed word per thread: element e of the word (magnitude bit 16 (e % 2) + e / 2, sign
// bit 8 above it) moves to magnitude bit 4 (e % 8) + 1 - e / 8 and sign bit 4 (e % 8) + 3 - e / 8.
__global__ __launch_bounds__(256) void repack_fp4_kernel(const uint32_t* __restrict__ codes, int64_t words,
                                                         uint32_t* __restrict__ out) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= words) return;
    const uint32_t w = codes[i];
    uint32_t o = 0;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
        const uint32_t m = (w >> (16 * (e & 1) + (e >> 1))) & 1u;
        const uint32_t s = (w >> (16 * (e & 1) + 8 + (e >> 1))) & 1u;
        const int j = e & 7, r = e >> 3;
        o |= (m << (4 * j + 1 - r)) | (s << (4 * j + 3 - r));
    }
    out[i] = o;
}

template <int BM, int BN, int WAVES_M, int WAVES_N, int STAGES>
hipError_t launch_fp8_cfg(const ConvFp8Args& args, hipStream_t stream) {
    ConvFp8Args a = args;
    const int64_t M = (int64_t)a.N * a.P * a.Q;
    const int64_t tilesN = (a.K + BN - 1) / BN;
    const int64_t tiles = ((M + BM - 1) / BM) * tilesN;
    if (tiles >= 0x7FFFFFFFll) return hipErrorInvalidValue;
    a.div_tilesN = make_fastdiv((uint32_t)tilesN);
    uint64_t rep = 0;
    for (int r = 0; r < a.R; ++r) rep |= 1ull << (r * a.S);
    a.rep_lo = (uint32_t)rep;
    a.rep_hi = (uint32_t)(rep >> 32);
    const dim3 grid((unsigned)tiles);
    if (a.C % BK == 0)
        hipLaunchKernelGGL((conv_fp8_kernel<BM, BN, WAVES_M, WAVES_N, STAGES, true>), grid, dim3(256), 0, stream, a);
    else
        hipLaunchKernelGGL((conv_fp8_kernel<BM, BN, WAVES_M, WAVES_N, STAGES, false>), grid, dim3(256), 0, stream, a);
    return hipGetLastError();
}

}  // namespace

bool conv_fp8_eligible(const ConvFp8Args& a) {
    const int64_t n = (int64_t)a.R * a.S * a.C;
    const int64_t xbytes = (int64_t)a.N * a.H * a.W * a.C;
    const int64_t cbytes = (int64_t)((a.K + 63) / 64) * ((n + 63) / 64) * 1024;
    return a.C % 16 == 0 && a.R * a.S <= 63 && xbytes < 0x7FFFFFF0ll && cbytes < 0x7FFFFFF0ll;
}

int conv_fp8_tile(const ConvFp8Args& a) {
    const int forced = knob(KNOB_FP8_TILE);
    if (forced >= 1 && forced <= 4) return forced;
    const int64_t M = (int64_t)a.N * a.P * a.Q;
    int cfg = a.K > 128 ? 1 : (a.K > 64 ? 2 : 3);
    const int bm = 128, bn = cfg == 1 ? 256 : (cfg == 2 ? 128 : 64);
    // too few tiles for one wave of blocks: 64-pixel x 128-filter tiles
    if (((M + bm - 1) / bm) * ((a.K + bn - 1) / bn) < 384 && a.K >= 128) cfg = 4;
    return cfg;
}

hipError_t launch_conv_fp8(const ConvFp8Args& args, hipStream_t stream) {
    if (!conv_fp8_eligible(args)) return hipErrorInvalidValue;
    ConvFp8Args a = args;
    a.div_q = make_fastdiv((uint32_t)a.Q);
    a.div_pq = make_fastdiv((uint32_t)a.P * (uint32_t)a.Q);
    switch (conv_fp8_tile(a)) {
        case 2: return launch_fp8_cfg<128, 128, 2, 2, 3>(a, stream);
        case 3: return launch_fp8_cfg<128, 64, 2, 2, 3>(a, stream);
        case 4: return launch_fp8_cfg<64, 128, 1, 4, 4>(a, stream);
        default: return launch_fp8_cfg<128, 256, 1, 4, 3>(a, stream);
    }
}

hipError_t launch_quantize_act_fp8(const void* x, int x_f32, int64_t count, float inv, uint8_t* q,
                                   hipStream_t stream) {
    const int64_t threads = (count + 15) / 16;
    const int64_t blocks = (threads + 255) / 256;
    if (blocks >= 0x7FFFFFFFll) return hipErrorInvalidValue;
    if (x_f32)
        hipLaunchKernelGGL(quantize_act_fp8_kernel<true>, dim3((unsigned)blocks), dim3(256), 0, stream, x, count, inv, q);
    else
        hipLaunchKernelGGL(quantize_act_fp8_kernel<false>, dim3((unsigned)blocks), dim3(256), 0, stream, x, count, inv, q);
    return hipGetLastError();
}

hipError_t launch_repack_fp4(const uint32_t* codes, int64_t words, uint32_t* out, hipStream_t stream) {
    const int64_t blocks = (words + 255) / 256;
    if (blocks >= 0x7FFFFFFFll) return hipErrorInvalidValue;
    hipLaunchKernelGGL(repack_fp4_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, codes, words, out);
    return hipGetLastError();
}

}  // namespace tbn
