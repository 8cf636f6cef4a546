// tbn_kernels.h -- host-side launchers of the gfx950 kernels (internal to libtbn).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>

#include "tbn.h"

namespace tbn {

// Test and tuning knobs (tbn_tuning.h); -1 = unset, the built-in choice.
enum Knob { KNOB_CONV_TILE = 0, KNOB_CONV_SPLITS = 1, KNOB_WGRAD_CFG = 2, KNOB_WGRAD_PIX = 3, KNOB_WGRAD_PF = 4,
            KNOB_I8_TILE = 5, KNOB_FC_VARIANT = 6, KNOB_FP8_TILE = 7 };
int knob(int which);

// Record the detail of an error for tbn_last_error() on this thread; returns s.
tbn_status set_error(tbn_status s, const std::string& what);

// Unsigned division by a runtime constant d >= 1 for numerators below 2^31
// (round-up multiplier: q = (mulhi(n, mul) + n) >> shift).
struct FastDiv {
    uint32_t d, mul, shift;
};

inline FastDiv make_fastdiv(uint32_t d) {
    FastDiv f;
    f.d = d;
    uint32_t s = 0;
    while ((1ull << s) < d) ++s;
    f.shift = s;
    f.mul = (uint32_t)(((1ull << 32) * ((1ull << s) - d)) / d + 1);
    return f;
}

__device__ __forceinline__ uint32_t fdiv(uint32_t n, const FastDiv& f) {
    return (__umulhi(n, f.mul) + n) >> f.shift;
}

// Geometry + operands of the implicit GEMM that serves both the forward pass and the
// backward-data pass.  Rows are output pixels (n, p, q) of an NHWC "input" x; columns
// are the Kf "filters" whose packed codes hold n = R*S*C elements each.
struct ConvGemmArgs {
    const void* x;            // NHWC [N][H][W][C], bf16 (or fp32 when x_f32)
    const uint32_t* codes;    // TBN2 codes of Kf filters of n elements
    const uint32_t* apair;    // per element pair: bf16 scale pair (backward-data), or null
    const float* colscale;    // per column fp32 scale (alpha in the forward pass), or null
    const float* scale;       // epilogue: optional per-column multiplier
    const float* bias;        // epilogue: optional per-column addend
    const void* residual;     // epilogue: optional NHWC [N][P][Q][Kf] addend, y's dtype
    void* y;                  // NHWC [N][P][Q][Kf]
    int32_t N, H, W, C, Kf, R, S, sh, sw, ph, pw, P, Q;
    int32_t relu;
    int32_t x_f32;
    int32_t y_f32;
    // LDS-DMA kernel: write y with non-temporal (streaming) stores -- set by its launcher
    // for outputs too large to be read back from the last-level cache
    int32_t y_stream;
    FastDiv div_q, div_pq;    // division by Q and by P*Q (output pixel -> (n, p, q))
    float* partial;           // split-K: fp32 partial sums [splits][M][Kf] (workspace)
    int32_t splits;           // split-K: number of reduction ranges (1 = none)
    int32_t chunks_per_split; // split-K: 64-element stages per range
    // LDS-DMA kernel: division by the tile count and by the column-tile count (the block
    // index -> (split, tile) -> (row tile, column tile) maps), and the 64-bit pattern
    // sum_{r < R} 2^(r*S) that replicates a filter row's in-image taps over its rows
    FastDiv div_tiles, div_tilesN;
    uint32_t rep_lo, rep_hi;
    // thin-input kernel only: real-valued filters [Kf][R][S][C] fp32 (rounded to bf16 as
    // they are staged) in place of the packed codes, for a layer kept in full precision
    const float* wdense;
};

hipError_t launch_quantize(const float* w, int64_t K, int64_t n, uint32_t* codes, float* alpha,
                           int32_t* counts, hipStream_t stream);

// Momentum-SGD operands of the fused update-and-quantise step ([K][n] fp32 each).
struct SgdArgs {
    float* w;
    float* v;
    const float* g;
    float lr, mu, wd;
};
hipError_t launch_sgd_quantize(const SgdArgs& sgd, int64_t K, int64_t n, uint32_t* codes, float* alpha,
                               int32_t* counts, hipStream_t stream);

// Discretisation variant: thr_bits = bit pattern of the magnitude threshold t > 0 (1.0f is
// Eq. 3), uni = per-weight uniform numbers in [0, 1) for stochastic discretisation (null:
// deterministic).
struct QuantVariant {
    uint32_t thr_bits;
    const float* uni;
};
hipError_t launch_quantize_variant(const float* w, int64_t K, int64_t n, const QuantVariant& var, uint32_t* codes,
                                   float* alpha, int32_t* counts, hipStream_t stream);

hipError_t launch_conv_gemm(const ConvGemmArgs& a, hipStream_t stream);

// LDS-DMA variant (bf16 x, C % 8 == 0, R*S <= 63, x < 2 GiB).  Its plan picks the tile
// shape and, for layers with too few output tiles to fill the GPU, a split of the reduction
// whose fp32 partials live in caller workspace; cfg >= 10 forces a tile shape.
struct ConvPlan {
    int cfg;
    int splits;
    int chunks_per_split;
    size_t partial_bytes;
};
bool conv_dma_eligible(const ConvGemmArgs& a);
ConvPlan plan_conv_dma(const ConvGemmArgs& a, int cfg);
hipError_t launch_conv_dma(const ConvGemmArgs& a, const ConvPlan& plan, hipStream_t stream);
// Tile-shape and reduction-split overrides for tuning and tests (the knobs of
// tbn_tuning.h, read once per call; -1 when unset).
int conv_tile_override();
int conv_splits_override();
// Bytes of split-K partials the forward / backward-data GEMM of these arguments needs.
size_t conv_gemm_partial_bytes(const ConvGemmArgs& a);

// Forward pass for inputs with few channels (C < 8 bf16, or fp32 with C <= 8): input patch
// and decoded filters staged in LDS with the channels padded to a power of two.
struct ThinGeom {
    int32_t CP, T, logT, RT, WPITCH, PH, PW;
    int32_t tiles_p, tiles_q;
    int64_t ntiles;
    int32_t w_off, p_off, s_off, lds_bytes;
    int32_t pbuf;  // bf16 elements per patch buffer (two buffers)
    int32_t rowlen, nelem, ept;  // input elements per patch row, per patch, per thread
    FastDiv div_rowlen, div_c;
    FastDiv div_pqt, div_tq;  // tile index -> (image, tile row, tile column); ntiles < 2^31
    // large inputs: the input is first written once into workspace as a zero-bordered NHWC
    // copy with CP channels [N][Hp][Wp][CP] bf16, from which every patch is a block of whole
    // 16-byte pieces copied straight into LDS (ppr pieces per patch row, npieces per patch,
    // ni copy instructions per wave)
    int32_t dma, Hp, Wp, ppr, npieces, ni;
    int64_t ws_bytes;
};
bool conv_thin_plan(const ConvGemmArgs& a, ThinGeom* g);
// Direct fp32-FMA kernel for small forward layers (at most 147 filter elements, C <= 8).
bool conv_direct_eligible(const ConvGemmArgs& a);
hipError_t launch_conv_direct(const ConvGemmArgs& a, hipStream_t stream);
hipError_t launch_conv_thin(const ConvGemmArgs& a, const ThinGeom& g, hipStream_t stream);

// Forward pass of a fully-connected layer (the filter window covers the whole input map)
// for a batch of at most 16: codes streamed from HBM into 16x16x32 MFMAs.
struct FcStreamPlan {
    int32_t n, nsteps, xpitch, lds_bytes;
    int32_t variant;  // loads in flight per wave (tuning knob; 0 = built-in)
};
bool fc_stream_plan(const ConvGemmArgs& a, FcStreamPlan* p);
hipError_t launch_fc_stream(const ConvGemmArgs& a, const FcStreamPlan& p, hipStream_t stream);

// Re-pack the codes of K filters [K][R][S][C] into the codes of the C filters of the
// transposed, spatially flipped layer [C][R][S][K] (backward-data operand), and build
// the bf16 scale pairs of that layer's element pairs; filters Kreal..K-1 (channel padding
// of the gradient) get scale 0.
hipError_t launch_repack_bwd(const uint32_t* codes, const float* alpha, int32_t K, int32_t Kreal, int32_t R,
                             int32_t S, int32_t C, uint32_t* codes_t, uint32_t* apair, hipStream_t stream);

struct WgradArgs {
    const uint16_t* x;        // NHWC [N][H][W][C] bf16
    const uint16_t* dy;       // NHWC [N][P][Q][K] bf16
    float* out;               // [splits][K][R*S*C] fp32 partials, or dw when splits == 1
    int32_t N, H, W, C, K, R, S, sh, sw, ph, pw, P, Q;
    int32_t splits;           // number of reduction splits (grid y)
    int32_t chunks_per_split; // 64-pixel chunks per split
    int32_t accumulate;       // splits == 1 only: add to `out` instead of overwriting
};

hipError_t launch_wgrad(const WgradArgs& a, hipStream_t stream);

// LDS-DMA + transposing-read variant (C % 8 == 0, K % 8 == 0, tensors < 2 GiB),
// 256 x 256 output tiles of 512 threads; launch_wgrad uses it when eligible.
bool wgrad_dma_eligible(const WgradArgs& a);
// Stage layout of the LDS-DMA weight-gradient kernel (1 = pixel-major rows for K >= 128,
// 0 = segment-major; the stage-layout knob forces one for tests), its output tiles and how many
// blocks are resident at once.
struct WgradDmaPlan {
    int cfg, tiles, resident_blocks;
    int pix;  // pixel-major kernel: pixels per stage (32, 48 or 64)
};
WgradDmaPlan wgrad_dma_plan(int K, int J);
hipError_t launch_wgrad_dma(const WgradArgs& a, hipStream_t stream);

// Channel counts the LDS-DMA kernels cannot take (C < 8 inputs, K % 8 != 0 gradients): the
// tensor copied into Cp channels (a multiple of 8, zeros beyond C); for the filter gradient
// of a C < 8 input, the 8-channel gradient's split partials summed into the C-channel dw.
hipError_t launch_pad_channels(const uint16_t* x, int64_t pixels, int32_t C, int32_t Cp, uint16_t* xp,
                               hipStream_t stream);
hipError_t launch_split_reduce_compact(const float* partials, int32_t splits, int64_t rows, int32_t C, float* dw,
                                       int32_t accumulate, hipStream_t stream);
// partials [splits][stride]: dw[i] (+)= sum_z partials[z][i] for i < count
hipError_t launch_split_reduce(const float* partials, int32_t splits, int64_t count, int64_t stride, float* dw,
                               int32_t accumulate, hipStream_t stream);

// Forward pass on int8 activation codes (int8 MFMA): y = act(float(sum q * W~) *
// float(alpha_k * x_scale)), NHWC, bf16 or fp32 output.  Needs C % 16 == 0, R*S <= 63,
// int32-safe sums and tensors below 2 GiB (conv_i8_eligible); no workspace.
struct ConvI8Args {
    const int8_t* x;          // NHWC [N][H][W][C] int8 codes
    const uint32_t* codes;    // TBN2 codes of K filters of n = R*S*C elements
    const float* alpha;       // [K]
    void* y;                  // NHWC [N][P][Q][K]
    float x_scale;
    int32_t N, H, W, C, K, R, S, sh, sw, ph, pw, P, Q;
    int32_t relu, y_f32;
    FastDiv div_q, div_pq, div_tilesN;
    uint32_t rep_lo, rep_hi;  // sum_{r < R} 2^(r*S)
};
bool conv_i8_eligible(const ConvI8Args& a);
// Tile shape (1: 128 x 256, 2: 128 x 128, 3: 128 x 64, 4: 64 x 128); the int8 tile knob forces one.
int conv_i8_tile(const ConvI8Args& a);
hipError_t launch_conv_i8(const ConvI8Args& a, hipStream_t stream);
// q = clamp(round-half-even(x * inv), -127, 127), NaN -> 0; x bf16 or fp32.
hipError_t launch_quantize_act_i8(const void* x, int x_f32, int64_t count, float inv, int8_t* q,
                                  hipStream_t stream);

// Forward pass on E4M3 activation codes (scaled fp8 x E2M1 MFMA): y = act(sum f * W~ *
// fp32(alpha_k * x_scale)), the sum fp32, NHWC, bf16 or fp32 output.  The filters in the
// E2M1 operand layout (launch_repack_fp4).  Needs C % 16 == 0, R*S <= 63 and tensors below
// 2 GiB (conv_fp8_eligible); no workspace.
struct ConvFp8Args {
    const uint8_t* x;         // NHWC [N][H][W][C] E4M3 codes
    const uint32_t* codes;    // E2M1-layout codes of K filters of n = R*S*C elements
    const float* alpha;       // [K]
    void* y;                  // NHWC [N][P][Q][K]
    float x_scale;
    int32_t N, H, W, C, K, R, S, sh, sw, ph, pw, P, Q;
    int32_t relu, y_f32;
    FastDiv div_q, div_pq, div_tilesN;
    uint32_t rep_lo, rep_hi;  // sum_{r < R} 2^(r*S)
};
bool conv_fp8_eligible(const ConvFp8Args& a);
// Tile shape (1: 128 x 256, 2: 128 x 128, 3: 128 x 64, 4: 64 x 128); the fp8 tile knob forces one.
int conv_fp8_tile(const ConvFp8Args& a);
hipError_t launch_conv_fp8(const ConvFp8Args& a, hipStream_t stream);
// q = E4M3(fp32(x * inv)): nearest, ties to even, saturating at +-448, NaN -> 0; x bf16 or fp32.
hipError_t launch_quantize_act_fp8(const void* x, int x_f32, int64_t count, float inv, uint8_t* q,
                                   hipStream_t stream);
// The packed codes (`words` 32-bit words) rewritten in the E2M1 operand layout.
hipError_t launch_repack_fp4(const uint32_t* codes, int64_t words, uint32_t* out, hipStream_t stream);

struct DenseConvArgs {
    const void* x;
    const float* w;          // [K][R][S][C] fp32, rounded to bf16 on load
    const float* scale;
    const float* bias;
    const void* residual;
    void* y;
    int32_t N, H, W, C, K, R, S, sh, sw, ph, pw, P, Q;
    int32_t relu, x_f32, y_f32;
};

hipError_t launch_conv_dense(const DenseConvArgs& a, hipStream_t stream);

struct PoolArgs {
    int32_t N, H, W, C, k, s, pad, P, Q;
};

hipError_t launch_maxpool_fwd(const PoolArgs& a, const uint16_t* x, uint16_t* y, int32_t* arg, hipStream_t s);
hipError_t launch_maxpool_bwd(const PoolArgs& a, const uint16_t* dy, const int32_t* arg, void* dx, int dx_f32,
                              hipStream_t s);
hipError_t launch_avgpool(int32_t N, int32_t HW, int32_t C, const uint16_t* x, void* y, int y_f32, hipStream_t s);
// Batch normalisation statistics: per-chunk partial sums in workspace, then per channel.
struct BnPlan {
    int64_t rpc, chunks;  // rows per chunk, chunks
    int32_t slices;       // groups of 256 channel groups
    int32_t vec;          // C % 8 == 0: 8 channels per 16-byte access
    size_t ws_bytes;      // two fp32 partial arrays [chunks][C]
};
BnPlan plan_bn(int64_t rows, int32_t C);
hipError_t launch_bn_train_fwd(const uint16_t* x, int64_t rows, int32_t C, const float* gamma, const float* beta,
                               float eps, int relu, uint16_t* y, float* mean, float* inv_std, float* ws,
                               hipStream_t s);
hipError_t launch_bn_train_bwd(const uint16_t* x, const uint16_t* y, const uint16_t* dy, int64_t rows, int32_t C,
                               int relu, const float* mean, const float* inv_std, const float* gamma, float* dgamma,
                               float* dbeta, uint16_t* dx, float* ws, hipStream_t s);
hipError_t launch_relu_bwd(const uint16_t* y, const uint16_t* dy, int64_t total, uint16_t* dx, hipStream_t s);
hipError_t launch_softmax_xent(const float* z, const int32_t* labels, int32_t N, int32_t K, float* loss,
                               float* loss_per_sample, uint16_t* dz, hipStream_t s);

hipError_t launch_sgd(float* w, float* v, const float* g, int64_t count, float lr, float mu,
                      float wd, hipStream_t stream);

}  // namespace tbn
