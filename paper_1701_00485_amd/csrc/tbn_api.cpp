// tbn_api.cpp -- the C ABI of libtbn (declared in include/tbn.h): argument validation,
// shape arithmetic, workspace sizing and kernel launches on the caller's stream.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <cstring>
#include <string>

#include "tbn.h"
#include "tbn_kernels.h"

namespace {

thread_local std::string g_last_error;

tbn_status fail(tbn_status s, const char* what) {
    g_last_error = what;
    return s;
}

tbn_status hip_fail(hipError_t e, const char* where) {
    g_last_error = std::string(where) + ": " + hipGetErrorString(e);
    return TBN_ERR_HIP;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

constexpr int64_t kI32Max = 0x7FFFFFFF;

int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }

// a * b * c > limit, for positive factors, without overflowing
bool product_over(int64_t a, int64_t b, int64_t c, int64_t limit) {
    int64_t ab, abc;
    return __builtin_mul_overflow(a, b, &ab) || __builtin_mul_overflow(ab, c, &abc) || abc > limit;
}

struct Geometry {
    int64_t N, H, W, C, K, R, S, sh, sw, ph, pw, P, Q;
};

tbn_status check_desc(const tbn_conv_desc* d, Geometry* g) {
    if (!d) return fail(TBN_ERR_NULL, "desc is NULL");
    if (d->n <= 0 || d->h <= 0 || d->w <= 0 || d->c <= 0 || d->k <= 0 || d->r <= 0 || d->s <= 0)
        return fail(TBN_ERR_SHAPE, "every size must be positive");
    if (d->stride_h <= 0 || d->stride_w <= 0) return fail(TBN_ERR_SHAPE, "strides must be positive");
    if (d->pad_h < 0 || d->pad_w < 0) return fail(TBN_ERR_SHAPE, "padding must be non-negative");
    const int64_t hp = (int64_t)d->h + 2 * (int64_t)d->pad_h, wp = (int64_t)d->w + 2 * (int64_t)d->pad_w;
    if (hp < d->r || wp < d->s) return fail(TBN_ERR_SHAPE, "filter larger than the padded input");
    g->N = d->n; g->H = d->h; g->W = d->w; g->C = d->c; g->K = d->k; g->R = d->r; g->S = d->s;
    g->sh = d->stride_h; g->sw = d->stride_w; g->ph = d->pad_h; g->pw = d->pad_w;
    g->P = (hp - d->r) / d->stride_h + 1;
    g->Q = (wp - d->s) / d->stride_w + 1;
    // index arithmetic inside the kernels is 32-bit for pixels and filter elements (the
    // products are formed with overflow checks: each factor alone may be near 2^32)
    if (product_over(g->N, g->P, g->Q, kI32Max) || product_over(g->N, g->H, g->W, kI32Max))
        return fail(TBN_ERR_SHAPE, "more than 2^31 - 1 pixels");
    if (product_over(g->R, g->S, g->C, kI32Max / 2) || product_over(g->R, g->S, g->K, kI32Max / 2))
        return fail(TBN_ERR_SHAPE, "filter has more than 2^30 elements");
    return TBN_OK;
}

tbn::WgradArgs wgrad_args(const Geometry& g) {
    tbn::WgradArgs a = {};
    a.N = (int32_t)g.N; a.H = (int32_t)g.H; a.W = (int32_t)g.W; a.C = (int32_t)g.C; a.K = (int32_t)g.K;
    a.R = (int32_t)g.R; a.S = (int32_t)g.S; a.sh = (int32_t)g.sh; a.sw = (int32_t)g.sw;
    a.ph = (int32_t)g.ph; a.pw = (int32_t)g.pw; a.P = (int32_t)g.P; a.Q = (int32_t)g.Q;
    return a;
}

// bwd_weight: number of reduction splits for a geometry (shared by sizing and launch).
// The LDS-DMA kernel runs one 512-thread block per CU; the fallback four per CU.
int wgrad_splits(const Geometry& g) {
    const int64_t J = g.R * g.S * g.C;
    const bool dma = tbn::wgrad_dma_eligible(wgrad_args(g));
    const tbn::WgradDmaPlan plan = tbn::wgrad_dma_plan((int)g.K, (int)J);
    const int64_t tiles = dma ? plan.tiles : ((g.K + 127) / 128) * ((J + 127) / 128);
    const int64_t chunks = (g.N * g.P * g.Q + 63) / 64;
    const int64_t target = dma ? plan.resident_blocks : 1024;
    int64_t splits = target / tiles;
    // at least 16 chunks per split for the LDS-DMA kernel, 4 for the register-staged one
    // (its first-layer shapes have one output tile and a long reduction)
    const int64_t min_chunks = dma ? 16 : 4;
    const int64_t max_by_len = chunks / min_chunks > 0 ? chunks / min_chunks : 1;
    if (splits > max_by_len) splits = max_by_len;
    if (splits > 256) splits = 256;
    if (splits < 1) splits = 1;
    return (int)splits;
}

// bwd_weight of an input with C < 8 channels (and K % 8 == 0): run on the LDS-DMA kernel
// over the input copied into 8 channels.  Workspace: the 8-channel input, then the split
// partials of the 8-channel gradient.
bool wgrad_pad8(const Geometry& g, Geometry* g8) {
    if (g.C >= 8 || g.K % 8 != 0) return false;
    *g8 = g;
    g8->C = 8;
    if (g8->R * g8->S * 8 > kI32Max / 2) return false;
    return tbn::wgrad_dma_eligible(wgrad_args(*g8));
}

int64_t pad8_x_bytes(const Geometry& g) { return round_up(g.N * g.H * g.W * 16, 256); }

// A gradient with K % 8 != 0 channels (a 10-way classifier): dy copied into Kp = K rounded
// up to 8 channels (zeros beyond K) so that both backward passes run on the LDS-DMA
// kernels.  `gk` is the geometry with Kp filters.
bool grad_padk(const Geometry& g, Geometry* gk) {
    if (g.K % 8 == 0 || g.C % 8 != 0) return false;
    *gk = g;
    gk->K = round_up(g.K, 8);
    if (gk->R * gk->S * gk->K > kI32Max / 2) return false;
    return true;
}

int64_t padk_dy_bytes(const Geometry& gk) { return round_up(gk.N * gk.P * gk.Q * gk.K * 2, 256); }

struct BwdDataWs {
    int64_t codes_bytes, apair_off, apair_bytes, partial_off, partial_bytes, total;
};

tbn::ConvGemmArgs bwd_data_args(const Geometry& g, tbn_dtype dxt);

BwdDataWs bwd_data_ws(const Geometry& g) {
    BwdDataWs w;
    const int64_t nt = g.R * g.S * g.K;
    const int64_t nbt = (nt + 63) / 64;
    w.codes_bytes = ((g.C + 63) / 64) * nbt * 256 * 4;
    w.apair_off = round_up(w.codes_bytes, 256);
    w.apair_bytes = nbt * 32 * 4;
    w.partial_off = w.apair_off + round_up(w.apair_bytes, 256);
    // the split-K partials of the GEMM do not depend on the output dtype
    w.partial_bytes = (int64_t)tbn::conv_gemm_partial_bytes(bwd_data_args(g, TBN_BF16));
    w.total = w.partial_off + w.partial_bytes;
    return w;
}

// Forward GEMM arguments of a geometry (pointers filled in by the caller).
tbn::ConvGemmArgs fwd_args(const Geometry& g, tbn_dtype xt, tbn_dtype yt) {
    tbn::ConvGemmArgs a = {};
    a.N = (int32_t)g.N; a.H = (int32_t)g.H; a.W = (int32_t)g.W; a.C = (int32_t)g.C; a.Kf = (int32_t)g.K;
    a.R = (int32_t)g.R; a.S = (int32_t)g.S; a.sh = (int32_t)g.sh; a.sw = (int32_t)g.sw;
    a.ph = (int32_t)g.ph; a.pw = (int32_t)g.pw; a.P = (int32_t)g.P; a.Q = (int32_t)g.Q;
    a.x_f32 = xt == TBN_F32;
    a.y_f32 = yt == TBN_F32;
    return a;
}

// Backward-data as a forward convolution: dx = conv(dy, flipped transposed filter), padding
// R-1-pad, stride 1.
tbn::ConvGemmArgs bwd_data_args(const Geometry& g, tbn_dtype dxt) {
    tbn::ConvGemmArgs a = {};
    a.N = (int32_t)g.N; a.H = (int32_t)g.P; a.W = (int32_t)g.Q; a.C = (int32_t)g.K; a.Kf = (int32_t)g.C;
    a.R = (int32_t)g.R; a.S = (int32_t)g.S; a.sh = 1; a.sw = 1;
    a.ph = (int32_t)(g.R - 1 - g.ph); a.pw = (int32_t)(g.S - 1 - g.pw);
    a.P = (int32_t)g.H; a.Q = (int32_t)g.W;
    a.x_f32 = 0;
    a.y_f32 = dxt == TBN_F32;
    return a;
}

}  // namespace

namespace tbn {
tbn_status set_error(tbn_status s, const std::string& what) {
    g_last_error = what;
    return s;
}
}  // namespace tbn

extern "C" {

const char* tbn_status_str(tbn_status s) {
    switch (s) {
        case TBN_OK: return "TBN_OK";
        case TBN_ERR_NULL: return "TBN_ERR_NULL";
        case TBN_ERR_SHAPE: return "TBN_ERR_SHAPE";
        case TBN_ERR_UNSUPPORTED: return "TBN_ERR_UNSUPPORTED";
        case TBN_ERR_ALIGN: return "TBN_ERR_ALIGN";
        case TBN_ERR_WORKSPACE: return "TBN_ERR_WORKSPACE";
        case TBN_ERR_HIP: return "TBN_ERR_HIP";
    }
    return "TBN_ERR_UNKNOWN";
}

const char* tbn_last_error(void) { return g_last_error.c_str(); }

tbn_status tbn_conv_out_dims(const tbn_conv_desc* desc, int32_t* p, int32_t* q) {
    Geometry g;
    tbn_status st = check_desc(desc, &g);
    if (st != TBN_OK) return st;
    if (!p || !q) return fail(TBN_ERR_NULL, "output pointer is NULL");
    *p = (int32_t)g.P;
    *q = (int32_t)g.Q;
    return TBN_OK;
}

int64_t tbn_packed_words(int64_t k, int64_t n) {
    if (k <= 0 || n <= 0) return -1;
    return ((k + 63) / 64) * ((n + 63) / 64) * 256;
}

int64_t tbn_packed_row_words(int64_t n) {
    if (n <= 0) return -1;
    return (n + 63) / 64 * 4;
}

int64_t tbn_packed_bytes(int64_t k, int64_t n) {
    const int64_t w = tbn_packed_words(k, n);
    return w < 0 ? -1 : 4 * w;
}

tbn_status tbn_workspace_size(tbn_op op, const tbn_conv_desc* desc, size_t* bytes) {
    Geometry g;
    tbn_status st = check_desc(desc, &g);
    if (st != TBN_OK) return st;
    if (!bytes) return fail(TBN_ERR_NULL, "bytes is NULL");
    switch (op) {
        case TBN_OP_FWD: {
            // the same geometry may take another path for fp32 input: size for both
            const size_t b16 = tbn::conv_gemm_partial_bytes(fwd_args(g, TBN_BF16, TBN_BF16));
            const size_t b32 = tbn::conv_gemm_partial_bytes(fwd_args(g, TBN_F32, TBN_BF16));
            *bytes = b16 > b32 ? b16 : b32;
            return TBN_OK;
        }
        case TBN_OP_BWD_DATA: {
            Geometry gk;
            *bytes = grad_padk(g, &gk) ? (size_t)(round_up(bwd_data_ws(gk).total, 256) + padk_dy_bytes(gk))
                                       : (size_t)bwd_data_ws(g).total;
            return TBN_OK;
        }
        case TBN_OP_BWD_WEIGHT: {
            Geometry g8;
            if (wgrad_pad8(g, &g8)) {
                *bytes = (size_t)pad8_x_bytes(g) + (size_t)wgrad_splits(g8) * (size_t)(g.K * g.R * g.S * 8) * 4;
                return TBN_OK;
            }
            if (grad_padk(g, &g8) && tbn::wgrad_dma_eligible(wgrad_args(g8))) {
                *bytes = (size_t)padk_dy_bytes(g8) + (size_t)wgrad_splits(g8) * (size_t)(g8.K * g.R * g.S * g.C) * 4;
                return TBN_OK;
            }
            const int splits = wgrad_splits(g);
            *bytes = splits > 1 ? (size_t)splits * (size_t)(g.K * g.R * g.S * g.C) * 4 : 0;
            return TBN_OK;
        }
    }
    return fail(TBN_ERR_UNSUPPORTED, "unknown op");
}

tbn_status tbn_quantize(const float* w, int64_t k, int64_t n, uint32_t* codes, float* alpha, int32_t* counts,
                        hipStream_t stream) {
    if (!w || !codes || !alpha) return fail(TBN_ERR_NULL, "w, codes and alpha are required");
    if (k <= 0 || n <= 0) return fail(TBN_ERR_SHAPE, "k and n must be positive");
    if (n > kI32Max || k > kI32Max / 2) return fail(TBN_ERR_SHAPE, "k or n too large");
    if (!aligned4(w) || !aligned16(codes) || !aligned4(alpha) || (counts && !aligned4(counts)))
        return fail(TBN_ERR_ALIGN, "misaligned pointer");
    hipError_t e = tbn::launch_quantize(w, k, n, codes, alpha, counts, stream);
    return e == hipSuccess ? TBN_OK : hip_fail(e, "tbn_quantize");
}

tbn_status tbn_quantize_variant(const float* w, int64_t k, int64_t n, float threshold, const float* uniform,
                                uint32_t* codes, float* alpha, int32_t* counts, hipStream_t stream) {
    if (!w || !codes || !alpha) return fail(TBN_ERR_NULL, "w, codes and alpha are required");
    if (k <= 0 || n <= 0) return fail(TBN_ERR_SHAPE, "k and n must be positive");
    if (n > kI32Max || k > kI32Max / 2) return fail(TBN_ERR_SHAPE, "k or n too large");
    if (!(threshold > 0.0f) || !(threshold < 3.4028235e38f))
        return fail(TBN_ERR_SHAPE, "threshold must be positive and finite");
    if (uniform && threshold != 1.0f)
        return fail(TBN_ERR_UNSUPPORTED, "stochastic discretisation uses the threshold 1");
    if (!aligned4(w) || !aligned16(codes) || !aligned4(alpha) || (counts && !aligned4(counts)) ||
        (uniform && !aligned4(uniform)))
        return fail(TBN_ERR_ALIGN, "misaligned pointer");
    uint32_t thr_bits;
    memcpy(&thr_bits, &threshold, 4);
    hipError_t e = tbn::launch_quantize_variant(w, k, n, tbn::QuantVariant{thr_bits, uniform}, codes, alpha, counts,
                                                stream);
    return e == hipSuccess ? TBN_OK : hip_fail(e, "tbn_quantize_variant");
}

tbn_status tbn_conv2d_fwd(const tbn_conv_desc* desc, const void* x, tbn_dtype xt, const uint32_t* codes,
                          const float* alpha, const tbn_epilogue* ep, void* y, tbn_dtype yt, void* ws,
                          size_t ws_bytes, hipStream_t stream) {
    Geometry g;
    tbn_status st = check_desc(desc, &g);
    if (st != TBN_OK) return st;
    if (!x || !codes || !alpha || !y) return fail(TBN_ERR_NULL, "x, codes, alpha and y are required");
    if ((xt != TBN_BF16 && xt != TBN_F32) || (yt != TBN_BF16 && yt != TBN_F32))
        return fail(TBN_ERR_UNSUPPORTED, "unknown dtype");
    if (!aligned16(x) || !aligned16(codes) || !aligned16(y) || !aligned4(alpha))
        return fail(TBN_ERR_ALIGN, "x, codes and y must be 16-byte aligned");
    tbn::ConvGemmArgs a = fwd_args(g, xt, yt);
    const size_t need = tbn::conv_gemm_partial_bytes(a);
    if (need) {
        if (!ws || ws_bytes < need) return fail(TBN_ERR_WORKSPACE, "workspace too small");
        if (!aligned16(ws)) return fail(TBN_ERR_ALIGN, "workspace must be 16-byte aligned");
        a.partial = reinterpret_cast<float*>(ws);
    }
    a.x = x;
    a.codes = codes;
    a.apair = nullptr;
    a.colscale = alpha;
    if (ep) {
        if ((ep->scale && !aligned4(ep->scale)) || (ep->bias && !aligned4(ep->bias)) ||
            (ep->residual && !aligned16(ep->residual)))
            return fail(TBN_ERR_ALIGN, "misaligned epilogue pointer");
        a.scale = ep->scale;
        a.bias = ep->bias;
        a.residual = ep->residual;
        a.relu = ep->relu ? 1 : 0;
    }
    a.y = y;
    hipError_t e = tbn::launch_conv_gemm(a, stream);
    return e == hipSuccess ? TBN_OK : hip_fail(e, "tbn_conv2d_fwd");
}

tbn_status tbn_conv2d_fwd_dense(const tbn_conv_desc* desc, const void* x, tbn_dtype xt, const float* w,
                                const tbn_epilogue* ep, void* y, tbn_dtype yt, hipStream_t stream) {
    Geometry g;
    tbn_status st = check_desc(desc, &g);
    if (st != TBN_OK) return st;
    if (!x || !w || !y) return fail(TBN_ERR_NULL, "x, w and y are required");
    if ((xt != TBN_BF16 && xt != TBN_F32) || (yt != TBN_BF16 && yt != TBN_F32))
        return fail(TBN_ERR_UNSUPPORTED, "unknown dtype");
    if (!aligned16(x) || !aligned16(y) || !aligned4(w)) return fail(TBN_ERR_ALIGN, "misaligned pointer");
    if (g.K > 65535 * 16) return fail(TBN_ERR_SHAPE, "too many filters");
    tbn::DenseConvArgs a = {};
    if (ep) {
        if ((ep->scale && !aligned4(ep->scale)) || (ep->bias && !aligned4(ep->bias)) ||
            (ep->residual && !aligned16(ep->residual)))
            return fail(TBN_ERR_ALIGN, "misaligned epilogue pointer");
        a.scale = ep->scale;
        a.bias = ep->bias;
        a.residual = ep->residual;
        a.relu = ep->relu ? 1 : 0;
    }
    a.x = x;
    a.w = w;
    a.y = y;
    a.N = (int32_t)g.N; a.H = (int32_t)g.H; a.W = (int32_t)g.W; a.C = (int32_t)g.C; a.K = (int32_t)g.K;
    a.R = (int32_t)g.R; a.S = (int32_t)g.S; a.sh = (int32_t)g.sh; a.sw = (int32_t)g.sw;
    a.ph = (int32_t)g.ph; a.pw = (int32_t)g.pw; a.P = (int32_t)g.P; a.Q = (int32_t)g.Q;
    a.x_f32 = xt == TBN_F32;
    a.y_f32 = yt == TBN_F32;
    // few input channels: the thin-input MFMA kernel with the real filters staged as bf16
    // (inputs small enough to need no workspace); otherwise the vector-ALU kernel
    tbn::ConvGemmArgs t = fwd_args(g, xt, yt);
    t.x = x;
    t.wdense = w;
    t.scale = a.scale;
    t.bias = a.bias;
    t.residual = a.residual;
    t.relu = a.relu;
    t.y = y;
    tbn::ThinGeom tg;
    hipError_t e;
    if (tbn::conv_thin_plan(t, &tg) && !tg.dma)
        e = tbn::launch_conv_thin(t, tg, stream);
    else
        e = tbn::launch_conv_dense(a, stream);
    return e == hipSuccess ? TBN_OK : hip_fail(e, "tbn_conv2d_fwd_dense");
}

tbn_status tbn_conv2d_bwd_data(const tbn_conv_desc* desc, const void* dy, const uint32_t* codes, const float* alpha,
                               void* dx, tbn_dtype dxt, void* ws, size_t ws_bytes, hipStream_t stream) {
    Geometry g;
    tbn_status st = check_desc(desc, &g);
    if (st != TBN_OK) return st;
    if (!dy || !codes || !alpha || !dx) return fail(TBN_ERR_NULL, "dy, codes, alpha and dx are required");
    if (dxt != TBN_BF16 && dxt != TBN_F32) return fail(TBN_ERR_UNSUPPORTED, "unknown dtype");
    if (g.sh != 1 || g.sw != 1) return fail(TBN_ERR_UNSUPPORTED, "backward-data supports stride 1 only");
    if (!aligned16(dy) || !aligned16(codes) || !aligned16(dx) || !aligned4(alpha))
        return fail(TBN_ERR_ALIGN, "dy, codes and dx must be 16-byte aligned");
    // K % 8 != 0: the GEMM runs over dy copied into Kp channels (workspace, after the rest)
    Geometry gk;
    const bool padk = grad_padk(g, &gk);
    const Geometry& gg = padk ? gk : g;
    const BwdDataWs w = bwd_data_ws(gg);
    const int64_t dy_off = round_up(w.total, 256);  // the Kp-channel copy of dy (padk only)
    const int64_t total = padk ? dy_off + padk_dy_bytes(gk) : w.total;
    if (!ws || ws_bytes < (size_t)total) return fail(TBN_ERR_WORKSPACE, "workspace too small");
    if (!aligned16(ws)) return fail(TBN_ERR_ALIGN, "workspace must be 16-byte aligned");
    uint32_t* codes_t = reinterpret_cast<uint32_t*>(ws);
    uint32_t* apair = reinterpret_cast<uint32_t*>(reinterpret_cast<char*>(ws) + w.apair_off);
    hipError_t e = tbn::launch_repack_bwd(codes, alpha, (int32_t)gg.K, (int32_t)g.K, (int32_t)g.R, (int32_t)g.S,
                                          (int32_t)g.C, codes_t, apair, stream);
    if (e != hipSuccess) return hip_fail(e, "tbn_conv2d_bwd_data (repack)");
    const void* dyk = dy;
    if (padk) {
        uint16_t* dyp = reinterpret_cast<uint16_t*>(reinterpret_cast<char*>(ws) + dy_off);
        e = tbn::launch_pad_channels(reinterpret_cast<const uint16_t*>(dy), g.N * g.P * g.Q, (int32_t)g.K,
                                     (int32_t)gk.K, dyp, stream);
        if (e != hipSuccess) return hip_fail(e, "tbn_conv2d_bwd_data (channel copy)");
        dyk = dyp;
    }
    tbn::ConvGemmArgs a = bwd_data_args(gg, dxt);
    a.x = dyk;
    a.codes = codes_t;
    a.apair = apair;
    a.colscale = nullptr;
    a.y = dx;
    if (w.partial_bytes) a.partial = reinterpret_cast<float*>(reinterpret_cast<char*>(ws) + w.partial_off);
    e = tbn::launch_conv_gemm(a, stream);
    return e == hipSuccess ? TBN_OK : hip_fail(e, "tbn_conv2d_bwd_data");
}

tbn_status tbn_conv2d_bwd_weight(const tbn_conv_desc* desc, const void* x, const void* dy, float* dw,
                                 int32_t accumulate, void* ws, size_t ws_bytes, hipStream_t stream) {
    Geometry g;
    tbn_status st = check_desc(desc, &g);
    if (st != TBN_OK) return st;
    if (!x || !dy || !dw) return fail(TBN_ERR_NULL, "x, dy and dw are required");
    if (!aligned16(x) || !aligned16(dy) || !aligned16(dw)) return fail(TBN_ERR_ALIGN, "misaligned pointer");
    Geometry g8;
    if (wgrad_pad8(g, &g8)) {
        // few input channels: 8-channel copy of x, 8-channel gradient, channels < C kept
        const int splits = wgrad_splits(g8);
        const int64_t xb = pad8_x_bytes(g);
        const size_t need = (size_t)xb + (size_t)splits * (size_t)(g.K * g.R * g.S * 8) * 4;
        if (!ws || ws_bytes < need) return fail(TBN_ERR_WORKSPACE, "workspace too small");
        if (!aligned16(ws)) return fail(TBN_ERR_ALIGN, "workspace must be 16-byte aligned");
        uint16_t* x8 = reinterpret_cast<uint16_t*>(ws);
        float* part = reinterpret_cast<float*>(reinterpret_cast<uint8_t*>(ws) + xb);
        hipError_t e = tbn::launch_pad_channels(reinterpret_cast<const uint16_t*>(x), g.N * g.H * g.W, (int32_t)g.C, 8,
                                                x8, stream);
        if (e != hipSuccess) return hip_fail(e, "tbn_conv2d_bwd_weight (channel copy)");
        tbn::WgradArgs a = wgrad_args(g8);
        a.x = x8;
        a.dy = reinterpret_cast<const uint16_t*>(dy);
        a.out = part;
        const int64_t chunks = (g.N * g.P * g.Q + 63) / 64;
        a.splits = splits;
        a.chunks_per_split = (int32_t)((chunks + splits - 1) / splits);
        a.accumulate = 0;
        e = tbn::launch_wgrad(a, stream);
        if (e != hipSuccess) return hip_fail(e, "tbn_conv2d_bwd_weight");
        e = tbn::launch_split_reduce_compact(part, splits, g.K * g.R * g.S, (int32_t)g.C, dw, accumulate, stream);
        return e == hipSuccess ? TBN_OK : hip_fail(e, "tbn_conv2d_bwd_weight (reduce)");
    }
    if (grad_padk(g, &g8) && tbn::wgrad_dma_eligible(wgrad_args(g8))) {
        // K % 8 != 0: dy copied into Kp channels; rows k < K of the Kp-row partials summed
        const int splits = wgrad_splits(g8);
        const int64_t dyb = padk_dy_bytes(g8);
        const int64_t J = g.R * g.S * g.C;
        const size_t need = (size_t)dyb + (size_t)splits * (size_t)(g8.K * J) * 4;
        if (!ws || ws_bytes < need) return fail(TBN_ERR_WORKSPACE, "workspace too small");
        if (!aligned16(ws)) return fail(TBN_ERR_ALIGN, "workspace must be 16-byte aligned");
        uint16_t* dyp = reinterpret_cast<uint16_t*>(ws);
        float* part = reinterpret_cast<float*>(reinterpret_cast<uint8_t*>(ws) + dyb);
        hipError_t e = tbn::launch_pad_channels(reinterpret_cast<const uint16_t*>(dy), g.N * g.P * g.Q, (int32_t)g.K,
                                                (int32_t)g8.K, dyp, stream);
        if (e != hipSuccess) return hip_fail(e, "tbn_conv2d_bwd_weight (channel copy)");
        tbn::WgradArgs a = wgrad_args(g8);
        a.x = reinterpret_cast<const uint16_t*>(x);
        a.dy = dyp;
        a.out = part;
        const int64_t chunks = (g.N * g.P * g.Q + 63) / 64;
        a.splits = splits;
        a.chunks_per_split = (int32_t)((chunks + splits - 1) / splits);
        a.accumulate = 0;
        e = tbn::launch_wgrad(a, stream);
        if (e != hipSuccess) return hip_fail(e, "tbn_conv2d_bwd_weight");
        e = tbn::launch_split_reduce(part, splits, g.K * J, g8.K * J, dw, accumulate, stream);
        return e == hipSuccess ? TBN_OK : hip_fail(e, "tbn_conv2d_bwd_weight (reduce)");
    }
    const int splits = wgrad_splits(g);
    const int64_t count = g.K * g.R * g.S * g.C;
    const bool direct = splits == 1;  // one split writes (or adds to) dw itself
    if (!direct) {
        const size_t need = (size_t)splits * (size_t)count * 4;
        if (!ws || ws_bytes < need) return fail(TBN_ERR_WORKSPACE, "workspace too small");
        if (!aligned16(ws)) return fail(TBN_ERR_ALIGN, "workspace must be 16-byte aligned");
    }
    tbn::WgradArgs a = wgrad_args(g);
    a.x = reinterpret_cast<const uint16_t*>(x);
    a.dy = reinterpret_cast<const uint16_t*>(dy);
    a.out = direct ? dw : reinterpret_cast<float*>(ws);
    const int64_t chunks = (g.N * g.P * g.Q + 63) / 64;
    a.splits = splits;
    a.chunks_per_split = (int32_t)((chunks + splits - 1) / splits);
    a.accumulate = direct && accumulate ? 1 : 0;
    hipError_t e = tbn::launch_wgrad(a, stream);
    if (e != hipSuccess) return hip_fail(e, "tbn_conv2d_bwd_weight");
    if (!direct) {
        e = tbn::launch_split_reduce(reinterpret_cast<const float*>(ws), splits, count, count, dw, accumulate, stream);
        if (e != hipSuccess) return hip_fail(e, "tbn_conv2d_bwd_weight (reduce)");
    }
    return TBN_OK;
}

tbn_status tbn_sgd_step(float* w, float* v, const float* g, int64_t count, float lr, float momentum,
                        float weight_decay, hipStream_t stream) {
    if (!w || !v || !g) return fail(TBN_ERR_NULL, "w, v and g are required");
    if (count <= 0) return fail(TBN_ERR_SHAPE, "count must be positive");
    if (!aligned16(w) || !aligned16(v) || !aligned16(g)) return fail(TBN_ERR_ALIGN, "misaligned pointer");
    hipError_t e = tbn::launch_sgd(w, v, g, count, lr, momentum, weight_decay, stream);
    return e == hipSuccess ? TBN_OK : hip_fail(e, "tbn_sgd_step");
}

tbn_status tbn_sgd_step_quantize(float* w, float* v, const float* g, int64_t k, int64_t n, float lr,
                                 float momentum, float weight_decay, uint32_t* codes, float* alpha,
                                 int32_t* counts, hipStream_t stream) {
    if (!w || !v || !g || !codes || !alpha) return fail(TBN_ERR_NULL, "w, v, g, codes and alpha are required");
    if (k <= 0 || n <= 0) return fail(TBN_ERR_SHAPE, "k and n must be positive");
    if (n > kI32Max || k > kI32Max / 2) return fail(TBN_ERR_SHAPE, "k or n too large");
    if (!aligned4(w) || !aligned4(v) || !aligned4(g) || !aligned16(codes) || !aligned4(alpha) ||
        (counts && !aligned4(counts)))
        return fail(TBN_ERR_ALIGN, "misaligned pointer");
    const tbn::SgdArgs sgd = {w, v, g, lr, momentum, weight_decay};
    hipError_t e = tbn::launch_sgd_quantize(sgd, k, n, codes, alpha, counts, stream);
    return e == hipSuccess ? TBN_OK : hip_fail(e, "tbn_sgd_step_quantize");
}

tbn_status tbn_quantize_act_i8(const void* x, tbn_dtype xt, int64_t count, float inv_scale, int8_t* q,
                               hipStream_t stream) {
    if (!x || !q) return fail(TBN_ERR_NULL, "x and q are required");
    if (count <= 0) return fail(TBN_ERR_SHAPE, "count must be positive");
    if (count > ((int64_t)1 << 40)) return fail(TBN_ERR_SHAPE, "count too large");
    if (xt != TBN_BF16 && xt != TBN_F32) return fail(TBN_ERR_UNSUPPORTED, "unknown dtype");
    if (!(inv_scale > 0.0f) || inv_scale > 3.4028235e38f) return fail(TBN_ERR_SHAPE, "inv_scale must be finite and positive");
    if (!aligned16(x) || !aligned16(q)) return fail(TBN_ERR_ALIGN, "x and q must be 16-byte aligned");
    hipError_t e = tbn::launch_quantize_act_i8(x, xt == TBN_F32 ? 1 : 0, count, inv_scale, q, stream);
    return e == hipSuccess ? TBN_OK : hip_fail(e, "tbn_quantize_act_i8");
}

tbn_status tbn_conv2d_fwd_i8(const tbn_conv_desc* desc, const int8_t* x, const uint32_t* codes, const float* alpha,
                             float x_scale, int32_t relu, void* y, tbn_dtype yt, hipStream_t stream) {
    Geometry g;
    tbn_status st = check_desc(desc, &g);
    if (st != TBN_OK) return st;
    if (!x || !codes || !alpha || !y) return fail(TBN_ERR_NULL, "x, codes, alpha and y are required");
    if (yt != TBN_BF16 && yt != TBN_F32) return fail(TBN_ERR_UNSUPPORTED, "unknown dtype");
    if (!(x_scale == x_scale) || x_scale > 3.4028235e38f || x_scale < -3.4028235e38f)
        return fail(TBN_ERR_SHAPE, "x_scale must be finite");
    if (!aligned16(x) || !aligned16(codes) || !aligned16(y) || !aligned4(alpha))
        return fail(TBN_ERR_ALIGN, "x, codes and y must be 16-byte aligned");
    tbn::ConvI8Args a = {};
    a.x = x;
    a.codes = codes;
    a.alpha = alpha;
    a.y = y;
    a.x_scale = x_scale;
    a.N = (int32_t)g.N; a.H = (int32_t)g.H; a.W = (int32_t)g.W; a.C = (int32_t)g.C; a.K = (int32_t)g.K;
    a.R = (int32_t)g.R; a.S = (int32_t)g.S; a.sh = (int32_t)g.sh; a.sw = (int32_t)g.sw;
    a.ph = (int32_t)g.ph; a.pw = (int32_t)g.pw; a.P = (int32_t)g.P; a.Q = (int32_t)g.Q;
    a.relu = relu ? 1 : 0;
    a.y_f32 = yt == TBN_F32 ? 1 : 0;
    if (!tbn::conv_i8_eligible(a))
        return fail(TBN_ERR_UNSUPPORTED, "int8 forward needs C % 16 == 0, R*S <= 63, 254*R*S*C < 2^31 and tensors < 2 GiB");
    hipError_t e = tbn::launch_conv_i8(a, stream);
    return e == hipSuccess ? TBN_OK : hip_fail(e, "tbn_conv2d_fwd_i8");
}

tbn_status tbn_quantize_act_fp8(const void* x, tbn_dtype xt, int64_t count, float inv_scale, uint8_t* q,
                                hipStream_t stream) {
    if (!x || !q) return fail(TBN_ERR_NULL, "x and q are required");
    if (count <= 0) return fail(TBN_ERR_SHAPE, "count must be positive");
    if (count > ((int64_t)1 << 40)) return fail(TBN_ERR_SHAPE, "count too large");
    if (xt != TBN_BF16 && xt != TBN_F32) return fail(TBN_ERR_UNSUPPORTED, "unknown dtype");
    if (!(inv_scale > 0.0f) || inv_scale > 3.4028235e38f) return fail(TBN_ERR_SHAPE, "inv_scale must be finite and positive");
    if (!aligned16(x) || !aligned16(q)) return fail(TBN_ERR_ALIGN, "x and q must be 16-byte aligned");
    hipError_t e = tbn::launch_quantize_act_fp8(x, xt == TBN_F32 ? 1 : 0, count, inv_scale, q, stream);
    return e == hipSuccess ? TBN_OK : hip_fail(e, "tbn_quantize_act_fp8");
}

tbn_status tbn_repack_codes_fp4(const uint32_t* codes, int64_t words, uint32_t* out, hipStream_t stream) {
    if (!codes || !out) return fail(TBN_ERR_NULL, "codes and out are required");
    if (words <= 0 || words > ((int64_t)1 << 40)) return fail(TBN_ERR_SHAPE, "words must be positive");
    if (!aligned4(codes) || !aligned4(out)) return fail(TBN_ERR_ALIGN, "codes and out must be 4-byte aligned");
    const uintptr_t c0 = (uintptr_t)codes, o0 = (uintptr_t)out, nb = (uintptr_t)words * 4;
    if (c0 < o0 + nb && o0 < c0 + nb) return fail(TBN_ERR_SHAPE, "codes and out overlap");
    hipError_t e = tbn::launch_repack_fp4(codes, words, out, stream);
    return e == hipSuccess ? TBN_OK : hip_fail(e, "tbn_repack_codes_fp4");
}

tbn_status tbn_conv2d_fwd_fp8(const tbn_conv_desc* desc, const uint8_t* x, const uint32_t* codes, const float* alpha,
                              float x_scale, int32_t relu, void* y, tbn_dtype yt, hipStream_t stream) {
    Geometry g;
    tbn_status st = check_desc(desc, &g);
    if (st != TBN_OK) return st;
    if (!x || !codes || !alpha || !y) return fail(TBN_ERR_NULL, "x, codes, alpha and y are required");
    if (yt != TBN_BF16 && yt != TBN_F32) return fail(TBN_ERR_UNSUPPORTED, "unknown dtype");
    if (!(x_scale == x_scale) || x_scale > 3.4028235e38f || x_scale < -3.4028235e38f)
        return fail(TBN_ERR_SHAPE, "x_scale must be finite");
    if (!aligned16(x) || !aligned16(codes) || !aligned16(y) || !aligned4(alpha))
        return fail(TBN_ERR_ALIGN, "x, codes and y must be 16-byte aligned");
    tbn::ConvFp8Args a = {};
    a.x = x;
    a.codes = codes;
    a.alpha = alpha;
    a.y = y;
    a.x_scale = x_scale;
    a.N = (int32_t)g.N; a.H = (int32_t)g.H; a.W = (int32_t)g.W; a.C = (int32_t)g.C; a.K = (int32_t)g.K;
    a.R = (int32_t)g.R; a.S = (int32_t)g.S; a.sh = (int32_t)g.sh; a.sw = (int32_t)g.sw;
    a.ph = (int32_t)g.ph; a.pw = (int32_t)g.pw; a.P = (int32_t)g.P; a.Q = (int32_t)g.Q;
    a.relu = relu ? 1 : 0;
    a.y_f32 = yt == TBN_F32 ? 1 : 0;
    if (!tbn::conv_fp8_eligible(a))
        return fail(TBN_ERR_UNSUPPORTED, "fp8 forward needs C % 16 == 0, R*S <= 63 and tensors < 2 GiB");
    hipError_t e = tbn::launch_conv_fp8(a, stream);
    return e == hipSuccess ? TBN_OK : hip_fail(e, "tbn_conv2d_fwd_fp8");
}

namespace {

tbn_status check_pool(const tbn_pool_desc* d, tbn::PoolArgs* a) {
    if (!d) return fail(TBN_ERR_NULL, "desc is NULL");
    if (d->n <= 0 || d->h <= 0 || d->w <= 0 || d->c <= 0 || d->k <= 0 || d->stride <= 0 || d->pad < 0)
        return fail(TBN_ERR_SHAPE, "invalid pooling geometry");
    if (d->h + 2 * (int64_t)d->pad < d->k || d->w + 2 * (int64_t)d->pad < d->k)
        return fail(TBN_ERR_SHAPE, "window larger than the padded input");
    // the kernels index window rows and columns, and the argmax position h*W + w, in 32 bits
    if ((int64_t)d->h + 2 * (int64_t)d->pad + d->stride > kI32Max ||
        (int64_t)d->w + 2 * (int64_t)d->pad + d->stride > kI32Max || product_over(d->h, d->w, 1, kI32Max))
        return fail(TBN_ERR_SHAPE, "more than 2^31 - 1 positions per image");
    const int64_t P = ((int64_t)d->h + 2 * (int64_t)d->pad - d->k) / d->stride + 1;
    const int64_t Q = ((int64_t)d->w + 2 * (int64_t)d->pad - d->k) / d->stride + 1;
    if (product_over((int64_t)d->n * d->c, d->h, d->w, (int64_t)1 << 40) ||
        product_over((int64_t)d->n * d->c, P, Q, (int64_t)1 << 40))
        return fail(TBN_ERR_SHAPE, "tensor too large");
    a->N = d->n; a->H = d->h; a->W = d->w; a->C = d->c; a->k = d->k; a->s = d->stride; a->pad = d->pad;
    a->P = (int32_t)P;
    a->Q = (int32_t)Q;
    return TBN_OK;
}

}  // namespace

tbn_status tbn_pool_out_dims(const tbn_pool_desc* desc, int32_t* p, int32_t* q) {
    tbn::PoolArgs a;
    tbn_status st = check_pool(desc, &a);
    if (st != TBN_OK) return st;
    if (!p || !q) return fail(TBN_ERR_NULL, "output pointer is NULL");
    *p = a.P;
    *q = a.Q;
    return TBN_OK;
}

tbn_status tbn_maxpool2d_fwd(const tbn_pool_desc* desc, const void* x, void* y, int32_t* argmax, hipStream_t stream) {
    tbn::PoolArgs a;
    tbn_status st = check_pool(desc, &a);
    if (st != TBN_OK) return st;
    if (!x || !y) return fail(TBN_ERR_NULL, "x and y are required");
    if (!aligned16(x) || !aligned16(y) || (argmax && !aligned16(argmax))) return fail(TBN_ERR_ALIGN, "misaligned pointer");
    hipError_t e = tbn::launch_maxpool_fwd(a, reinterpret_cast<const uint16_t*>(x), reinterpret_cast<uint16_t*>(y),
                                           argmax, stream);
    return e == hipSuccess ? TBN_OK : hip_fail(e, "tbn_maxpool2d_fwd");
}

tbn_status tbn_maxpool2d_bwd(const tbn_pool_desc* desc, const void* dy, const int32_t* argmax, void* dx, tbn_dtype dxt,
                             hipStream_t stream) {
    tbn::PoolArgs a;
    tbn_status st = check_pool(desc, &a);
    if (st != TBN_OK) return st;
    if (!dy || !argmax || !dx) return fail(TBN_ERR_NULL, "dy, argmax and dx are required");
    if (dxt != TBN_BF16 && dxt != TBN_F32) return fail(TBN_ERR_UNSUPPORTED, "unknown dtype");
    if (!aligned16(dy) || !aligned16(dx) || !aligned16(argmax)) return fail(TBN_ERR_ALIGN, "misaligned pointer");
    hipError_t e = tbn::launch_maxpool_bwd(a, reinterpret_cast<const uint16_t*>(dy), argmax, dx, dxt == TBN_F32, stream);
    return e == hipSuccess ? TBN_OK : hip_fail(e, "tbn_maxpool2d_bwd");
}

tbn_status tbn_avgpool_global(int32_t n, int32_t h, int32_t w, int32_t c, const void* x, void* y, tbn_dtype yt,
                              hipStream_t stream) {
    if (!x || !y) return fail(TBN_ERR_NULL, "x and y are required");
    if (n <= 0 || h <= 0 || w <= 0 || c <= 0) return fail(TBN_ERR_SHAPE, "sizes must be positive");
    if (product_over(h, w, 1, kI32Max)) return fail(TBN_ERR_SHAPE, "more than 2^31 - 1 positions per image");
    if (product_over((int64_t)n * c, h, w, (int64_t)1 << 40)) return fail(TBN_ERR_SHAPE, "tensor too large");
    if (yt != TBN_BF16 && yt != TBN_F32) return fail(TBN_ERR_UNSUPPORTED, "unknown dtype");
    if (!aligned16(x) || !aligned16(y)) return fail(TBN_ERR_ALIGN, "misaligned pointer");
    hipError_t e = tbn::launch_avgpool(n, h * w, c, reinterpret_cast<const uint16_t*>(x), y, yt == TBN_F32, stream);
    return e == hipSuccess ? TBN_OK : hip_fail(e, "tbn_avgpool_global");
}

tbn_status tbn_batchnorm_workspace_size(int64_t rows, int32_t c, size_t* bytes) {
    if (!bytes) return fail(TBN_ERR_NULL, "bytes is NULL");
    if (rows <= 0 || c <= 0) return fail(TBN_ERR_SHAPE, "sizes must be positive");
    if (rows > kI32Max * (int64_t)64 || (int64_t)c > kI32Max / 64) return fail(TBN_ERR_SHAPE, "too large");
    *bytes = tbn::plan_bn(rows, c).ws_bytes;
    return TBN_OK;
}

static tbn_status check_bn_ws(int64_t rows, int32_t c, const void* ws, size_t ws_bytes) {
    if (!ws || ws_bytes < tbn::plan_bn(rows, c).ws_bytes) return fail(TBN_ERR_WORKSPACE, "workspace too small");
    if (!aligned16(ws)) return fail(TBN_ERR_ALIGN, "workspace must be 16-byte aligned");
    return TBN_OK;
}

tbn_status tbn_batchnorm_train_fwd(const void* x, int64_t rows, int32_t c, const float* gamma, const float* beta,
                                   float eps, int32_t relu, void* y, float* mean, float* inv_std, void* ws,
                                   size_t ws_bytes, hipStream_t stream) {
    if (!x || !gamma || !beta || !y || !mean || !inv_std) return fail(TBN_ERR_NULL, "missing pointer");
    if (rows <= 0 || c <= 0) return fail(TBN_ERR_SHAPE, "sizes must be positive");
    if (!aligned16(x) || !aligned16(y)) return fail(TBN_ERR_ALIGN, "misaligned pointer");
    tbn_status st = check_bn_ws(rows, c, ws, ws_bytes);
    if (st != TBN_OK) return st;
    hipError_t e = tbn::launch_bn_train_fwd(reinterpret_cast<const uint16_t*>(x), rows, c, gamma, beta, eps, relu ? 1 : 0,
                                            reinterpret_cast<uint16_t*>(y), mean, inv_std,
                                            reinterpret_cast<float*>(ws), stream);
    return e == hipSuccess ? TBN_OK : hip_fail(e, "tbn_batchnorm_train_fwd");
}

tbn_status tbn_batchnorm_train_bwd(const void* x, const void* y, const void* dy, int64_t rows, int32_t c, int32_t relu,
                                   const float* mean, const float* inv_std, const float* gamma, float* dgamma,
                                   float* dbeta, void* dx, void* ws, size_t ws_bytes, hipStream_t stream) {
    if (!x || !y || !dy || !mean || !inv_std || !gamma || !dgamma || !dbeta || !dx)
        return fail(TBN_ERR_NULL, "missing pointer");
    if (rows <= 0 || c <= 0) return fail(TBN_ERR_SHAPE, "sizes must be positive");
    if (!aligned16(x) || !aligned16(y) || !aligned16(dy) || !aligned16(dx)) return fail(TBN_ERR_ALIGN, "misaligned pointer");
    tbn_status st = check_bn_ws(rows, c, ws, ws_bytes);
    if (st != TBN_OK) return st;
    hipError_t e = tbn::launch_bn_train_bwd(reinterpret_cast<const uint16_t*>(x), reinterpret_cast<const uint16_t*>(y),
                                            reinterpret_cast<const uint16_t*>(dy), rows, c, relu ? 1 : 0, mean, inv_std,
                                            gamma, dgamma, dbeta, reinterpret_cast<uint16_t*>(dx),
                                            reinterpret_cast<float*>(ws), stream);
    return e == hipSuccess ? TBN_OK : hip_fail(e, "tbn_batchnorm_train_bwd");
}

tbn_status tbn_relu_bwd(const void* y, const void* dy, int64_t count, void* dx, hipStream_t stream) {
    if (!y || !dy || !dx) return fail(TBN_ERR_NULL, "missing pointer");
    if (count <= 0) return fail(TBN_ERR_SHAPE, "count must be positive");
    hipError_t e = tbn::launch_relu_bwd(reinterpret_cast<const uint16_t*>(y), reinterpret_cast<const uint16_t*>(dy), count,
                                        reinterpret_cast<uint16_t*>(dx), stream);
    return e == hipSuccess ? TBN_OK : hip_fail(e, "tbn_relu_bwd");
}

tbn_status tbn_softmax_xent(const float* logits, const int32_t* labels, int32_t n, int32_t classes, float* loss,
                            float* loss_per_sample, void* dlogits, hipStream_t stream) {
    if (!logits || !labels || !loss || !loss_per_sample || !dlogits) return fail(TBN_ERR_NULL, "missing pointer");
    if (n <= 0 || classes <= 0) return fail(TBN_ERR_SHAPE, "sizes must be positive");
    hipError_t e = tbn::launch_softmax_xent(logits, labels, n, classes, loss, loss_per_sample,
                                            reinterpret_cast<uint16_t*>(dlogits), stream);
    return e == hipSuccess ? TBN_OK : hip_fail(e, "tbn_softmax_xent");
}

}  // extern "C"
