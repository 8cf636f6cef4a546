/*
 * tbn_oracle.c -- plain, slow, fp64 CPU oracle for the Two-Bit Networks hot path
 * (Meng, Gu, Zhang, Wu, "Two-Bit Networks for Deep Learning on Resource-Constrained
 * Embedded Devices", arXiv 1701.00485).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the checker, not the product: only the test
 * suite, the smoke check and the CPU-baseline leg of the benchmark may load it.  It
 * shares no code, header, table or helper with the GPU library; the only thing both
 * sides see is the seeded input arrays.
 *
 * Every routine is the plain definition of what it computes, written with direct loops
 * in double precision, in the order the paper states the steps:
 *   - discretisation                      : Sec. 2, Eq. (3)
 *   - optimal per-filter scale            : Sec. 2, Eq. (4)-(5)
 *   - approximate convolution             : Sec. 2, Eq. (1); Sec. 3, Algorithm 1 (forward)
 *   - backward passes through the approximate filters, gradient w.r.t. the approximate
 *     filter used as the real-weight gradient : Sec. 3 (text) and Algorithm 1 (backward,
 *     update)
 *   - SGD with momentum and weight decay  : Sec. 4 (training set-up)
 *   - integer-activation forward variant  : Eq. (1) with the input replaced by int8 codes
 *     times one scale (an extension; see orc_conv_fwd_i8)
 *   - fp8-activation forward variant      : the same with E4M3 fp8 activation values (an
 *     extension; see orc_conv_fwd_fp8)
 * The 2-bit packed layout is this project's own storage format (the paper only says the
 * four values fit in two bits, abstract and Sec. 1); its definition is restated next to
 * the packer below.
 *
 * Pins: every function here is checked by the CPU test suite against something other
 * than itself (closed forms, library routines on special cases, brute force, adjoint
 * identities); none is "parity unpinned".
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_OK 0
#define ORC_ERR_NONFINITE 1
#define ORC_ERR_SHAPE 2

/* ------------------------------------------------------------------------------------ */
/* Rounding of an fp32 value to bf16, round-to-nearest-even on the 16 dropped bits      */
/* (IEEE 754 rounding rule applied to the bfloat16 format: 1 sign, 8 exponent, 7        */
/* fraction bits).  Used where a GPU operand is an fp32 input rounded to bf16 on load.   */
/* ------------------------------------------------------------------------------------ */
static double orc_round_bf16_one(float f) {
    uint32_t u;
    memcpy(&u, &f, 4);
    if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu) != 0) {
        return (double)f; /* NaN stays NaN */
    }
    uint32_t keep = u >> 16;
    uint32_t dropped = u & 0xFFFFu;
    if (dropped > 0x8000u || (dropped == 0x8000u && (keep & 1u))) keep += 1u;
    uint32_t r = keep << 16;
    float out;
    memcpy(&out, &r, 4);
    return (double)out;
}

void orc_round_bf16(const float* in, int64_t count, double* out) {
    for (int64_t i = 0; i < count; ++i) out[i] = orc_round_bf16_one(in[i]);
}

/* ------------------------------------------------------------------------------------ */
/* Sec. 2, Eq. (3): deterministic discretisation of one real weight.                    */
/*   -2 if W < -1;  -1 if -1 <= W <= 0;  1 if 0 < W <= 1;  2 if W > 1.                  */
/* ------------------------------------------------------------------------------------ */
static int orc_discretize_one(double w) {
    if (w < -1.0) return -2;
    if (w <= 0.0) return -1; /* here -1 <= w <= 0 */
    if (w <= 1.0) return 1;  /* here 0 < w <= 1 */
    return 2;                /* here w > 1 */
}

/*
 * Eq. (3) codes of the fp32 values whose bit patterns are start, start + 1, ...,
 * start + count - 1 (taken modulo 2^32), for the exhaustive check of the discretisation
 * over every fp32 value.  A NaN is outside the method and gets the marker 0.
 */
void orc_codes_of_bits(uint64_t start, int64_t count, int8_t* codes) {
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < count; ++i) {
        const uint32_t b = (uint32_t)(start + (uint64_t)i);
        float f;
        memcpy(&f, &b, sizeof f);
        codes[i] = isnan(f) ? 0 : (int8_t)orc_discretize_one((double)f);
    }
}

/*
 * Quantise K filters of n real weights each (w is [K][n], row k = filter k).
 * Writes codes [K][n] in {-2,-1,1,2}, the optimal scale alpha [K] (fp64, and its
 * single round-to-nearest fp32 value), the sizes |B1|, |B2| and the sums over B1 and
 * B2 of |W_i| for every filter.
 *   Eq. (3) gives the codes; Eq. (4) names the sets B1 = {|W_i| <= 1}, B2 = {|W_i| > 1};
 *   Eq. (5): alpha* = (sum_{B1}|W_i| + 2 sum_{B2}|W_i|) / (|B1| + 4|B2|).
 * Non-finite weights are outside the method's domain: the call returns
 * ORC_ERR_NONFINITE and writes nothing for that filter.
 * The sums run in index order in fp64.
 */
int orc_quantize(const float* w, int64_t K, int64_t n, int8_t* codes, double* alpha64,
                 float* alpha32, int64_t* b1_size, int64_t* b2_size, double* b1_sum,
                 double* b2_sum) {
    if (K < 0 || n <= 0) return ORC_ERR_SHAPE;
    int status = ORC_OK;
    for (int64_t k = 0; k < K; ++k) {
        const float* wk = w + k * n;
        int finite = 1;
        for (int64_t i = 0; i < n; ++i)
            if (!isfinite(wk[i])) finite = 0;
        if (!finite) {
            status = ORC_ERR_NONFINITE;
            continue;
        }
        /* Step 1 (Eq. 3): the two-bit filter. */
        for (int64_t i = 0; i < n; ++i) codes[k * n + i] = (int8_t)orc_discretize_one((double)wk[i]);
        /* Step 2 (Eq. 4-5): the optimal scale given the two-bit filter. */
        int64_t nb1 = 0, nb2 = 0;
        double s1 = 0.0, s2 = 0.0;
        for (int64_t i = 0; i < n; ++i) {
            double mag = fabs((double)wk[i]);
            if (mag <= 1.0) {
                nb1 += 1;
                s1 += mag;
            } else {
                nb2 += 1;
                s2 += mag;
            }
        }
        double a = (s1 + 2.0 * s2) / (double)(nb1 + 4 * nb2);
        if (alpha64) alpha64[k] = a;
        if (alpha32) alpha32[k] = (float)a; /* one round-to-nearest-even to fp32 */
        if (b1_size) b1_size[k] = nb1;
        if (b2_size) b2_size[k] = nb2;
        if (b1_sum) b1_sum[k] = s1;
        if (b2_sum) b2_sum[k] = s2;
    }
    return status;
}

/* Discretisation variants (Sec. 2 adopts the deterministic rule "for simplicity"):
 *   threshold t > 0 (uniform == NULL): the rule of Eq. (3) with the magnitude boundary at t
 *     instead of 1: -2 if W < -t, -1 if -t <= W <= 0, 1 if 0 < W <= t, 2 if W > t;
 *   uniform != NULL (t must be 1): stochastic rounding of a = clamp(W, -2, 2) to one of its
 *     two neighbouring levels among {-2, -1, 1, 2}, the upper one with probability equal
 *     to the distance from the lower one over the gap, so that E[code] = a.  Every decision
 *     is an fp32 comparison of the given uniform number u in [0, 1).
 * The scale is the minimiser of J(alpha) = ||W - alpha W~||^2 (Eq. 4) for the chosen codes:
 * dJ/dalpha = 0 gives alpha = sum_i W_i W~_i / sum_i W~_i^2, which for the deterministic
 * rules equals Eq. (5).  Sums in fp64 in index order, one rounding to fp32. */
static int orc_stochastic_one(float w, float u) {
    float a = fminf(fmaxf(w, -2.0f), 2.0f);
    if (a > 1.0f) return (u < a - 1.0f) ? 2 : 1;
    if (a < -1.0f) return (u < -1.0f - a) ? -2 : -1;
    return (u + u < a + 1.0f) ? 1 : -1;
}

int orc_quantize_variant(const float* w, int64_t K, int64_t n, float t, const float* uniform,
                         int8_t* codes, double* alpha64, float* alpha32, int64_t* b1_size,
                         int64_t* b2_size) {
    if (K < 0 || n <= 0 || !(t > 0.0f) || (uniform && t != 1.0f)) return ORC_ERR_SHAPE;
    int status = ORC_OK;
    for (int64_t k = 0; k < K; ++k) {
        const float* wk = w + k * n;
        int finite = 1;
        for (int64_t i = 0; i < n; ++i)
            if (!isfinite(wk[i])) finite = 0;
        if (!finite) {
            status = ORC_ERR_NONFINITE;
            continue;
        }
        double num = 0.0;
        int64_t nb1 = 0, nb2 = 0;
        for (int64_t i = 0; i < n; ++i) {
            const float x = wk[i];
            int c;
            if (uniform) {
                c = orc_stochastic_one(x, uniform[k * n + i]);
            } else if (x < -t) {
                c = -2;
            } else if (x <= 0.0f) {
                c = -1;
            } else if (x <= t) {
                c = 1;
            } else {
                c = 2;
            }
            codes[k * n + i] = (int8_t)c;
            num += (double)x * (double)c;
            if (c == 2 || c == -2) nb2 += 1; else nb1 += 1;
        }
        const double a = num / (double)(nb1 + 4 * nb2);
        if (alpha64) alpha64[k] = a;
        if (alpha32) alpha32[k] = (float)a;
        if (b1_size) b1_size[k] = nb1;
        if (b2_size) b2_size[k] = nb2;
    }
    return status;
}

/* ------------------------------------------------------------------------------------ */
/* Two-bit packed storage (this project's format; the paper fixes only that the four     */
/* values fit in two bits).                                                              */
/*   Filters are grouped in blocks of 64, reduction elements (index i of W^k_i, ordered  */
/*   (r, s, c) with c fastest) in blocks of 64.  With NB = ceil(n/64) and                */
/*   KB = ceil(K/64) the array holds KB*NB*64*4 words; element (k, i) lives in word      */
/*        ((k/64 * NB + i/64) * 64 + k%64) * 4 + (i%64)/16.                              */
/*   Inside a word, element e = i%16 uses j = e/2 and h = e%2:                           */
/*        bit 16h + j      = 1 iff |code| = 2  (the "magnitude" plane)                   */
/*        bit 16h + 8 + j  = 1 iff code < 0    (the "sign" plane).                       */
/*   Bits of filters k >= K and of elements i >= n are zero.                             */
/* ------------------------------------------------------------------------------------ */
int64_t orc_packed_words(int64_t K, int64_t n) {
    int64_t kb = (K + 63) / 64, nb = (n + 63) / 64;
    return kb * nb * 64 * 4;
}

int orc_pack(const int8_t* codes, int64_t K, int64_t n, uint32_t* words) {
    if (K <= 0 || n <= 0) return ORC_ERR_SHAPE;
    int64_t nb = (n + 63) / 64;
    memset(words, 0, (size_t)orc_packed_words(K, n) * sizeof(uint32_t));
    for (int64_t k = 0; k < K; ++k) {
        for (int64_t i = 0; i < n; ++i) {
            int c = codes[k * n + i];
            if (c != -2 && c != -1 && c != 1 && c != 2) return ORC_ERR_SHAPE;
            int64_t widx = ((k / 64 * nb + i / 64) * 64 + k % 64) * 4 + (i % 64) / 16;
            int e = (int)(i % 16), j = e / 2, h = e % 2;
            uint32_t bits = 0;
            if (c == 2 || c == -2) bits |= 1u << (16 * h + j);
            if (c < 0) bits |= 1u << (16 * h + 8 + j);
            words[widx] |= bits;
        }
    }
    return ORC_OK;
}

int orc_unpack(const uint32_t* words, int64_t K, int64_t n, int8_t* codes) {
    if (K <= 0 || n <= 0) return ORC_ERR_SHAPE;
    int64_t nb = (n + 63) / 64;
    for (int64_t k = 0; k < K; ++k) {
        for (int64_t i = 0; i < n; ++i) {
            int64_t widx = ((k / 64 * nb + i / 64) * 64 + k % 64) * 4 + (i % 64) / 16;
            int e = (int)(i % 16), j = e / 2, h = e % 2;
            int mag = (words[widx] >> (16 * h + j)) & 1u;
            int neg = (words[widx] >> (16 * h + 8 + j)) & 1u;
            int v = mag ? 2 : 1;
            codes[k * n + i] = (int8_t)(neg ? -v : v);
        }
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------------------------ */
/* Convolution geometry.  d[] = {N, H, W, C, K, R, S, stride_h, stride_w, pad_h, pad_w}. */
/* Cross-correlation with zero padding, dilation 1, one group; output size               */
/* P = floor((H + 2 pad_h - R) / stride_h) + 1, likewise Q.  Activations are NHWC,       */
/* filters are [K][R][S][C] (so filter element i = (r*S + s)*C + c).                     */
/* ------------------------------------------------------------------------------------ */
enum { DN, DH, DW, DC, DK, DR, DS, DSH, DSW, DPH, DPW };

int orc_out_dims(const int32_t* d, int32_t* P, int32_t* Q) {
    for (int i = 0; i < 7; ++i)
        if (d[i] <= 0) return ORC_ERR_SHAPE;
    if (d[DSH] <= 0 || d[DSW] <= 0 || d[DPH] < 0 || d[DPW] < 0) return ORC_ERR_SHAPE;
    int32_t p = (d[DH] + 2 * d[DPH] - d[DR]) / d[DSH] + 1;
    int32_t q = (d[DW] + 2 * d[DPW] - d[DS]) / d[DSW] + 1;
    if (d[DH] + 2 * d[DPH] < d[DR] || d[DW] + 2 * d[DPW] < d[DS]) return ORC_ERR_SHAPE;
    *P = p;
    *Q = q;
    return ORC_OK;
}

/*
 * Forward pass of one two-bit layer: Eq. (1), I * (alpha W~) = (alpha I) (+) W~, and
 * Algorithm 1's forward step.  x is NHWC [N][H][W][C], codes [K][R][S][C] in
 * {-2,-1,1,2}, alpha [K]; y is NHWC [N][P][Q][K].
 *   form 0: y = alpha_k * sum x * W~           (scale after the multiplication-free sum)
 *   form 1: y = sum (alpha_k x) * W~           (the literal right-hand side of Eq. 1)
 *   form 2: y = sum x * (alpha_k W~)           (the approximate filter W^ of Algorithm 1)
 * All three are equal in exact arithmetic; the tests check they agree in fp64.
 */
int orc_conv_fwd(const int32_t* d, const double* x, const int8_t* codes, const double* alpha,
                 int form, double* y) {
    int32_t P, Q;
    if (orc_out_dims(d, &P, &Q) != ORC_OK) return ORC_ERR_SHAPE;
    const int64_t N = d[DN], H = d[DH], W = d[DW], C = d[DC], K = d[DK], R = d[DR], S = d[DS];
    const int64_t sh = d[DSH], sw = d[DSW], ph = d[DPH], pw = d[DPW];
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t nn = 0; nn < N; ++nn) {
        for (int64_t p = 0; p < P; ++p) {
            for (int64_t q = 0; q < Q; ++q) {
                for (int64_t k = 0; k < K; ++k) {
                    double acc = 0.0;
                    for (int64_t r = 0; r < R; ++r) {
                        int64_t h = p * sh - ph + r;
                        if (h < 0 || h >= H) continue; /* zero padding */
                        for (int64_t s = 0; s < S; ++s) {
                            int64_t w = q * sw - pw + s;
                            if (w < 0 || w >= W) continue;
                            const double* xp = x + ((nn * H + h) * W + w) * C;
                            const int8_t* cp = codes + ((k * R + r) * S + s) * C;
                            for (int64_t c = 0; c < C; ++c) {
                                if (form == 1)
                                    acc += (alpha[k] * xp[c]) * (double)cp[c];
                                else if (form == 2)
                                    acc += xp[c] * (alpha[k] * (double)cp[c]);
                                else
                                    acc += xp[c] * (double)cp[c];
                            }
                        }
                    }
                    y[((nn * P + p) * Q + q) * K + k] = (form == 0) ? alpha[k] * acc : acc;
                }
            }
        }
    }
    return ORC_OK;
}

/*
 * Forward convolution with real-valued filters (Eq. 1 with full-precision weights): the
 * layer that stays in full precision (the first convolution of the CIFAR-shaped network)
 * uses it.  w is [K][R][S][C].
 */
int orc_conv_fwd_dense(const int32_t* d, const double* x, const double* wts, double* y) {
    int32_t P, Q;
    if (orc_out_dims(d, &P, &Q) != ORC_OK) return ORC_ERR_SHAPE;
    const int64_t N = d[DN], H = d[DH], W = d[DW], C = d[DC], K = d[DK], R = d[DR], S = d[DS];
    const int64_t sh = d[DSH], sw = d[DSW], ph = d[DPH], pw = d[DPW];
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t nn = 0; nn < N; ++nn) {
        for (int64_t p = 0; p < P; ++p) {
            for (int64_t q = 0; q < Q; ++q) {
                for (int64_t k = 0; k < K; ++k) {
                    double acc = 0.0;
                    for (int64_t r = 0; r < R; ++r) {
                        int64_t h = p * sh - ph + r;
                        if (h < 0 || h >= H) continue;
                        for (int64_t s = 0; s < S; ++s) {
                            int64_t w = q * sw - pw + s;
                            if (w < 0 || w >= W) continue;
                            const double* xp = x + ((nn * H + h) * W + w) * C;
                            const double* wp = wts + ((k * R + r) * S + s) * C;
                            for (int64_t c = 0; c < C; ++c) acc += xp[c] * wp[c];
                        }
                    }
                    y[((nn * P + p) * Q + q) * K + k] = acc;
                }
            }
        }
    }
    return ORC_OK;
}

/*
 * Integer-activation variant of the forward pass (an extension: the paper keeps the
 * activations in full precision and motivates the two-bit filters by arithmetic that needs
 * no multiplier, Sec. 1).  The input I of Eq. (1) is replaced by s * q with q an int8 code
 * per activation and s one positive fp32 scale per tensor, chosen by the caller.
 *
 * Activation codes: v = x * inv in fp32 (inv = the caller's fp32 reciprocal of s), then
 * q = v rounded to the nearest integer, ties to even, limited to [-127, 127]; a NaN
 * activation gets q = 0.
 */
void orc_quantize_act_i8(const float* x, int64_t count, float inv, int8_t* q) {
    for (int64_t i = 0; i < count; ++i) {
        const float v = x[i] * inv; /* one fp32 rounding */
        if (isnan(v)) {
            q[i] = 0;
            continue;
        }
        float r = nearbyintf(v); /* default rounding mode: nearest, ties to even */
        if (r > 127.0f) r = 127.0f;
        if (r < -127.0f) r = -127.0f;
        q[i] = (int8_t)r;
    }
}

/*
 * Forward pass on int8 activation codes (Eq. 1 with I = s q and the scale applied after
 * the multiplication-free sum):  acc[n,p,q,k] = sum_{r,s,c} q[n, p*sh-ph+r, q*sw-pw+s, c]
 * * W~[k,r,s,c] in exact integer arithmetic (zero padding), then, in fp32,
 * y = float(acc) * (alpha_k * s) with the scale product rounded first, and max(y, 0) when
 * relu != 0.  acc (optional) receives the exact sums.
 */
int orc_conv_fwd_i8(const int32_t* d, const int8_t* xq, const int8_t* codes, const float* alpha, float s,
                    int relu, int64_t* acc_out, float* y) {
    int32_t P, Q;
    if (orc_out_dims(d, &P, &Q) != ORC_OK) return ORC_ERR_SHAPE;
    const int64_t N = d[DN], H = d[DH], W = d[DW], C = d[DC], K = d[DK], R = d[DR], S = d[DS];
    const int64_t sh = d[DSH], sw = d[DSW], ph = d[DPH], pw = d[DPW];
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t nn = 0; nn < N; ++nn) {
        for (int64_t p = 0; p < P; ++p) {
            for (int64_t q = 0; q < Q; ++q) {
                for (int64_t k = 0; k < K; ++k) {
                    int64_t acc = 0;
                    for (int64_t r = 0; r < R; ++r) {
                        const int64_t h = p * sh - ph + r;
                        if (h < 0 || h >= H) continue;
                        for (int64_t t = 0; t < S; ++t) {
                            const int64_t w = q * sw - pw + t;
                            if (w < 0 || w >= W) continue;
                            const int8_t* xp = xq + ((nn * H + h) * W + w) * C;
                            const int8_t* cp = codes + ((k * R + r) * S + t) * C;
                            for (int64_t c = 0; c < C; ++c) acc += (int64_t)xp[c] * (int64_t)cp[c];
                        }
                    }
                    const int64_t o = ((nn * P + p) * Q + q) * K + k;
                    const float scale = alpha[k] * s;
                    float v = (float)acc * scale;
                    if (relu && !(v > 0.0f)) v = 0.0f;
                    y[o] = v;
                    if (acc_out) acc_out[o] = acc;
                }
            }
        }
    }
    return ORC_OK;
}

/* The same at `count` flat output indices idx (into [N][P][Q][K]); y[i] for idx[i]. */
int orc_conv_fwd_i8_sampled(const int32_t* d, const int8_t* xq, const int8_t* codes, const float* alpha, float s,
                            int relu, const int64_t* idx, int64_t count, float* y) {
    int32_t P, Q;
    if (orc_out_dims(d, &P, &Q) != ORC_OK) return ORC_ERR_SHAPE;
    const int64_t N = d[DN], H = d[DH], W = d[DW], C = d[DC], K = d[DK], R = d[DR], S = d[DS];
    const int64_t sh = d[DSH], sw = d[DSW], ph = d[DPH], pw = d[DPW];
    for (int64_t i = 0; i < count; ++i)
        if (idx[i] < 0 || idx[i] >= N * P * Q * K) return ORC_ERR_SHAPE;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < count; ++i) {
        const int64_t o = idx[i];
        const int64_t k = o % K, q = (o / K) % Q, p = (o / (K * Q)) % P, nn = o / (K * Q * P);
        int64_t acc = 0;
        for (int64_t r = 0; r < R; ++r) {
            const int64_t h = p * sh - ph + r;
            if (h < 0 || h >= H) continue;
            for (int64_t t = 0; t < S; ++t) {
                const int64_t w = q * sw - pw + t;
                if (w < 0 || w >= W) continue;
                const int8_t* xp = xq + ((nn * H + h) * W + w) * C;
                const int8_t* cp = codes + ((k * R + r) * S + t) * C;
                for (int64_t c = 0; c < C; ++c) acc += (int64_t)xp[c] * (int64_t)cp[c];
            }
        }
        const float scale = alpha[k] * s;
        float v = (float)acc * scale;
        if (relu && !(v > 0.0f)) v = 0.0f;
        y[i] = v;
    }
    return ORC_OK;
}

/*
 * Eight-bit floating-point activation variant (an extension of the same kind as the int8
 * one above): the input I of Eq. (1) is replaced by s * f with f an fp8 value in the E4M3
 * format and the two-bit filter values used as they are (+-1 and +-2 are exact in any
 * binary floating-point format with a 1-bit fraction, e.g. the 4-bit E2M1 one).
 *
 * E4M3 (the "fn" variant: no infinities): bit 7 sign, bits 6..3 exponent field e with bias
 * 7, bits 2..0 fraction m.  e = 0: (-1)^sign * (m / 8) * 2^-6 (zero and subnormals);
 * e = 1..15: (-1)^sign * (1 + m / 8) * 2^(e - 7), except the two codes with e = 15, m = 7
 * (0x7F, 0xFF), which are NaN.  The largest finite magnitude is 1.75 * 2^8 = 448.
 */
double orc_fp8_value(uint8_t code) {
    const int sign = code >> 7, e = (code >> 3) & 15, m = code & 7;
    if (e == 15 && m == 7) return NAN;
    const double mag = e == 0 ? ldexp(m / 8.0, -6) : ldexp(1.0 + m / 8.0, e - 7);
    return sign ? -mag : mag;
}

/*
 * Activation code of one value: v = x * inv in fp32 (inv = the caller's fp32 reciprocal of
 * s), then the finite E4M3 value nearest to v, found by comparing v with every finite
 * non-negative code (ties: the code with an even last fraction bit, i.e. the even code);
 * |v| > 448 takes +-448 (saturation); the sign bit is the sign bit of v (so -0 and small
 * negative values that round to zero keep it); a NaN gets code 0.
 */
uint8_t orc_fp8_encode(float v) {
    if (isnan(v)) return 0;
    const uint8_t sign = signbit(v) ? 0x80 : 0x00;
    const double a = fabs((double)v);
    if (a > 448.0) return sign | 0x7E;
    int best = 0;
    double best_d = INFINITY;
    for (int c = 0; c < 0x7F; ++c) { /* 0x00 .. 0x7E: every finite non-negative code */
        const double dist = fabs(orc_fp8_value((uint8_t)c) - a);
        if (dist < best_d || (dist == best_d && (c & 1) == 0)) {
            best_d = dist;
            best = c;
        }
    }
    return sign | (uint8_t)best;
}

void orc_quantize_act_fp8(const float* x, int64_t count, float inv, uint8_t* q) {
    for (int64_t i = 0; i < count; ++i) q[i] = orc_fp8_encode(x[i] * inv); /* one fp32 rounding */
}

/*
 * Forward pass on fp8 activation codes (Eq. 1 with I = s f):
 *   y[n,p,q,k] = alpha_k * s * sum_{r,s,c} f[n, p*sh-ph+r, q*sw-pw+s, c] * W~[k,r,s,c]
 * (zero padding), in double precision: every product is exact and so is the sum (the terms
 * are multiples of 2^-9 below 2^10 in magnitude), then the two scales; max(y, 0) when
 * relu != 0.  A NaN activation code makes its outputs NaN.
 */
int orc_conv_fwd_fp8(const int32_t* d, const uint8_t* xq, const int8_t* codes, const float* alpha, float s,
                     int relu, double* y) {
    int32_t P, Q;
    if (orc_out_dims(d, &P, &Q) != ORC_OK) return ORC_ERR_SHAPE;
    const int64_t N = d[DN], H = d[DH], W = d[DW], C = d[DC], K = d[DK], R = d[DR], S = d[DS];
    const int64_t sh = d[DSH], sw = d[DSW], ph = d[DPH], pw = d[DPW];
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t nn = 0; nn < N; ++nn) {
        for (int64_t p = 0; p < P; ++p) {
            for (int64_t q = 0; q < Q; ++q) {
                for (int64_t k = 0; k < K; ++k) {
                    double acc = 0.0;
                    for (int64_t r = 0; r < R; ++r) {
                        const int64_t h = p * sh - ph + r;
                        if (h < 0 || h >= H) continue;
                        for (int64_t t = 0; t < S; ++t) {
                            const int64_t w = q * sw - pw + t;
                            if (w < 0 || w >= W) continue;
                            const uint8_t* xp = xq + ((nn * H + h) * W + w) * C;
                            const int8_t* cp = codes + ((k * R + r) * S + t) * C;
                            for (int64_t c = 0; c < C; ++c) acc += orc_fp8_value(xp[c]) * (double)cp[c];
                        }
                    }
                    double v = acc * (double)alpha[k] * (double)s;
                    if (relu && !(v > 0.0)) v = 0.0;
                    y[((nn * P + p) * Q + q) * K + k] = v;
                }
            }
        }
    }
    return ORC_OK;
}

/* The same at `count` flat output indices idx (into [N][P][Q][K]); y[i] for idx[i]. */
int orc_conv_fwd_fp8_sampled(const int32_t* d, const uint8_t* xq, const int8_t* codes, const float* alpha, float s,
                             int relu, const int64_t* idx, int64_t count, double* y) {
    int32_t P, Q;
    if (orc_out_dims(d, &P, &Q) != ORC_OK) return ORC_ERR_SHAPE;
    const int64_t N = d[DN], H = d[DH], W = d[DW], C = d[DC], K = d[DK], R = d[DR], S = d[DS];
    const int64_t sh = d[DSH], sw = d[DSW], ph = d[DPH], pw = d[DPW];
    for (int64_t i = 0; i < count; ++i)
        if (idx[i] < 0 || idx[i] >= N * P * Q * K) return ORC_ERR_SHAPE;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < count; ++i) {
        const int64_t o = idx[i];
        const int64_t k = o % K, q = (o / K) % Q, p = (o / (K * Q)) % P, nn = o / (K * Q * P);
        double acc = 0.0;
        for (int64_t r = 0; r < R; ++r) {
            const int64_t h = p * sh - ph + r;
            if (h < 0 || h >= H) continue;
            for (int64_t t = 0; t < S; ++t) {
                const int64_t w = q * sw - pw + t;
                if (w < 0 || w >= W) continue;
                const uint8_t* xp = xq + ((nn * H + h) * W + w) * C;
                const int8_t* cp = codes + ((k * R + r) * S + t) * C;
                for (int64_t c = 0; c < C; ++c) acc += orc_fp8_value(xp[c]) * (double)cp[c];
            }
        }
        double v = acc * (double)alpha[k] * (double)s;
        if (relu && !(v > 0.0)) v = 0.0;
        y[i] = v;
    }
    return ORC_OK;
}

/*
 * Backward pass to the layer input through the approximate filters W^ = alpha W~
 * (Sec. 3: both passes use the approximate filters; Algorithm 1, backward step).
 * By the chain rule through y[n,p,q,k] = sum x[n, p*sh-ph+r, q*sw-pw+s, c] W^[k,r,s,c]:
 *   dx[n,h,w,c] = sum over (p,q,k,r,s) with p*sh-ph+r = h, q*sw-pw+s = w of
 *                 W^[k,r,s,c] * dy[n,p,q,k]
 * written here as the scatter over every (n,p,q,k,r,s,c) term.
 */
int orc_conv_bwd_data(const int32_t* d, const double* dy, const int8_t* codes,
                      const double* alpha, double* dx) {
    int32_t P, Q;
    if (orc_out_dims(d, &P, &Q) != ORC_OK) return ORC_ERR_SHAPE;
    const int64_t N = d[DN], H = d[DH], W = d[DW], C = d[DC], K = d[DK], R = d[DR], S = d[DS];
    const int64_t sh = d[DSH], sw = d[DSW], ph = d[DPH], pw = d[DPW];
#pragma omp parallel for schedule(static)
    for (int64_t nn = 0; nn < N; ++nn) {
        double* dxn = dx + nn * H * W * C;
        for (int64_t i = 0; i < H * W * C; ++i) dxn[i] = 0.0;
        for (int64_t p = 0; p < P; ++p)
            for (int64_t q = 0; q < Q; ++q)
                for (int64_t k = 0; k < K; ++k) {
                    double g = dy[((nn * P + p) * Q + q) * K + k];
                    for (int64_t r = 0; r < R; ++r) {
                        int64_t h = p * sh - ph + r;
                        if (h < 0 || h >= H) continue;
                        for (int64_t s = 0; s < S; ++s) {
                            int64_t w = q * sw - pw + s;
                            if (w < 0 || w >= W) continue;
                            const int8_t* cp = codes + ((k * R + r) * S + s) * C;
                            double* o = dxn + (h * W + w) * C;
                            for (int64_t c = 0; c < C; ++c) o[c] += (alpha[k] * (double)cp[c]) * g;
                        }
                    }
                }
    }
    return ORC_OK;
}

/*
 * Gradient with respect to the approximate filter W^ (Algorithm 1, backward step):
 *   dW^[k,r,s,c] = sum_{n,p,q} dy[n,p,q,k] * x[n, p*sh-ph+r, q*sw-pw+s, c].
 * Sec. 3 updates the real-valued filters with this gradient unchanged (the real weights
 * are kept only to accumulate small updates), so it is also the real-weight gradient.
 */
int orc_conv_bwd_weight(const int32_t* d, const double* x, const double* dy, double* dw) {
    int32_t P, Q;
    if (orc_out_dims(d, &P, &Q) != ORC_OK) return ORC_ERR_SHAPE;
    const int64_t N = d[DN], H = d[DH], W = d[DW], C = d[DC], K = d[DK], R = d[DR], S = d[DS];
    const int64_t sh = d[DSH], sw = d[DSW], ph = d[DPH], pw = d[DPW];
#pragma omp parallel for schedule(static)
    for (int64_t k = 0; k < K; ++k) {
        double* dwk = dw + k * R * S * C;
        for (int64_t i = 0; i < R * S * C; ++i) dwk[i] = 0.0;
        for (int64_t nn = 0; nn < N; ++nn)
            for (int64_t p = 0; p < P; ++p)
                for (int64_t q = 0; q < Q; ++q) {
                    double g = dy[((nn * P + p) * Q + q) * K + k];
                    for (int64_t r = 0; r < R; ++r) {
                        int64_t h = p * sh - ph + r;
                        if (h < 0 || h >= H) continue;
                        for (int64_t s = 0; s < S; ++s) {
                            int64_t w = q * sw - pw + s;
                            if (w < 0 || w >= W) continue;
                            const double* xp = x + ((nn * H + h) * W + w) * C;
                            double* o = dwk + (r * S + s) * C;
                            for (int64_t c = 0; c < C; ++c) o[c] += g * xp[c];
                        }
                    }
                }
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------------------------ */
/* Sampled forms for layers too large for the full loops: each requested element is      */
/* computed on its own from the same definitions.  Index arrays are flat element         */
/* indices into the NHWC / KRSC output tensors.  The bf16-valued inputs arrive as        */
/* their raw 16-bit patterns (exact in fp64), so a full-size tensor need not be widened. */
/* ------------------------------------------------------------------------------------ */
static double orc_bf16_bits_to_double(uint16_t b) {
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, 4);
    return (double)f;
}

int orc_conv_fwd_sampled_bf16(const int32_t* d, const uint16_t* x, const int8_t* codes,
                              const double* alpha, const int64_t* idx, int64_t count,
                              double* out) {
    int32_t P, Q;
    if (orc_out_dims(d, &P, &Q) != ORC_OK) return ORC_ERR_SHAPE;
    const int64_t H = d[DH], W = d[DW], C = d[DC], K = d[DK], R = d[DR], S = d[DS];
    const int64_t sh = d[DSH], sw = d[DSW], ph = d[DPH], pw = d[DPW];
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t t = 0; t < count; ++t) {
        int64_t e = idx[t];
        int64_t k = e % K, q = (e / K) % Q, p = (e / (K * Q)) % P, nn = e / (K * Q * P);
        double acc = 0.0;
        for (int64_t r = 0; r < R; ++r) {
            int64_t h = p * sh - ph + r;
            if (h < 0 || h >= H) continue;
            for (int64_t s = 0; s < S; ++s) {
                int64_t w = q * sw - pw + s;
                if (w < 0 || w >= W) continue;
                const uint16_t* xp = x + ((nn * H + h) * W + w) * C;
                const int8_t* cp = codes + ((k * R + r) * S + s) * C;
                for (int64_t c = 0; c < C; ++c) acc += orc_bf16_bits_to_double(xp[c]) * (double)cp[c];
            }
        }
        out[t] = alpha[k] * acc;
    }
    return ORC_OK;
}

/* dx at chosen (n,h,w,c): the gather over every (k,r,s) whose output position
 * p = (h + ph - r)/sh, q = (w + pw - s)/sw is integral and inside the output. */
int orc_conv_bwd_data_sampled_bf16(const int32_t* d, const uint16_t* dy, const int8_t* codes,
                                   const double* alpha, const int64_t* idx, int64_t count,
                                   double* out) {
    int32_t P, Q;
    if (orc_out_dims(d, &P, &Q) != ORC_OK) return ORC_ERR_SHAPE;
    const int64_t H = d[DH], W = d[DW], C = d[DC], K = d[DK], R = d[DR], S = d[DS];
    const int64_t sh = d[DSH], sw = d[DSW], ph = d[DPH], pw = d[DPW];
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t t = 0; t < count; ++t) {
        int64_t e = idx[t];
        int64_t c = e % C, w = (e / C) % W, h = (e / (C * W)) % H, nn = e / (C * W * H);
        double acc = 0.0;
        for (int64_t r = 0; r < R; ++r) {
            int64_t ph_ = h + ph - r;
            if (ph_ < 0 || ph_ % sh != 0) continue;
            int64_t p = ph_ / sh;
            if (p >= P) continue;
            for (int64_t s = 0; s < S; ++s) {
                int64_t qw_ = w + pw - s;
                if (qw_ < 0 || qw_ % sw != 0) continue;
                int64_t q = qw_ / sw;
                if (q >= Q) continue;
                const uint16_t* g = dy + ((nn * P + p) * Q + q) * K;
                for (int64_t k = 0; k < K; ++k)
                    acc += (alpha[k] * (double)codes[((k * R + r) * S + s) * C + c]) *
                           orc_bf16_bits_to_double(g[k]);
            }
        }
        out[t] = acc;
    }
    return ORC_OK;
}

int orc_conv_bwd_weight_sampled_bf16(const int32_t* d, const uint16_t* x, const uint16_t* dy,
                                     const int64_t* idx, int64_t count, double* out) {
    int32_t P, Q;
    if (orc_out_dims(d, &P, &Q) != ORC_OK) return ORC_ERR_SHAPE;
    const int64_t N = d[DN], H = d[DH], W = d[DW], C = d[DC], K = d[DK], R = d[DR], S = d[DS];
    const int64_t sh = d[DSH], sw = d[DSW], ph = d[DPH], pw = d[DPW];
#pragma omp parallel for schedule(dynamic, 4)
    for (int64_t t = 0; t < count; ++t) {
        int64_t e = idx[t];
        int64_t c = e % C, s = (e / C) % S, r = (e / (C * S)) % R, k = e / (C * S * R);
        double acc = 0.0;
        for (int64_t nn = 0; nn < N; ++nn)
            for (int64_t p = 0; p < P; ++p) {
                int64_t h = p * sh - ph + r;
                if (h < 0 || h >= H) continue;
                for (int64_t q = 0; q < Q; ++q) {
                    int64_t w = q * sw - pw + s;
                    if (w < 0 || w >= W) continue;
                    acc += orc_bf16_bits_to_double(dy[((nn * P + p) * Q + q) * K + k]) *
                           orc_bf16_bits_to_double(x[((nn * H + h) * W + w) * C + c]);
                }
            }
        out[t] = acc;
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------------------------ */
/* Algorithm 1, parameter update, with the optimiser of Sec. 4: SGD with momentum mu and */
/* weight decay lambda (no dampening, no Nesterov term):                                 */
/*   v <- mu v + (g + lambda w);   w <- w - eta v.                                      */
/* g is the gradient with respect to the approximate filter, applied to the real weights.*/
/* ------------------------------------------------------------------------------------ */
void orc_sgd(double* w, double* v, const double* g, int64_t count, double eta, double mu,
             double lambda) {
    for (int64_t i = 0; i < count; ++i) {
        v[i] = mu * v[i] + (g[i] + lambda * w[i]);
        w[i] = w[i] - eta * v[i];
    }
}

/* The same two update lines in fp32, each multiply-add fused and rounded once (C99 fmaf).
 * The updated weight decides the next iteration's codes (Eq. 3), an integer result, so
 * the fused update-and-quantise step is checked against this form, which reproduces the
 * fp32 rounding of the update exactly; orc_sgd above is the same step in fp64. */
void orc_sgd_f32(float* w, float* v, const float* g, int64_t count, float eta, float mu,
                 float lambda) {
    for (int64_t i = 0; i < count; ++i) {
        v[i] = fmaf(mu, v[i], fmaf(lambda, w[i], g[i]));
        w[i] = fmaf(-eta, v[i], w[i]);
    }
}

/* ------------------------------------------------------------------------------------ */
/* Layers the workloads put around the two-bit convolutions (Sec. 4 uses ResNet-18 with  */
/* batch normalisation).  Textbook definitions, NHWC, fp64.                               */
/* ------------------------------------------------------------------------------------ */

/* Max pooling, window k x k, stride s, padding p (padded positions never win).  The
 * index of the maximum is the flat NHWC input index; ties go to the first maximum in
 * row-major window order.  Windows with no valid input produce 0 and index -1. */
int orc_maxpool_fwd(const int32_t* dims /* N,H,W,C,k,s,p */, const double* x, double* y,
                    int64_t* arg) {
    const int64_t N = dims[0], H = dims[1], W = dims[2], C = dims[3], k = dims[4], s = dims[5],
                  p = dims[6];
    if (N <= 0 || H <= 0 || W <= 0 || C <= 0 || k <= 0 || s <= 0 || p < 0 || H + 2 * p < k ||
        W + 2 * p < k)
        return ORC_ERR_SHAPE;
    const int64_t P = (H + 2 * p - k) / s + 1, Q = (W + 2 * p - k) / s + 1;
    for (int64_t n = 0; n < N; ++n)
        for (int64_t pp = 0; pp < P; ++pp)
            for (int64_t qq = 0; qq < Q; ++qq)
                for (int64_t c = 0; c < C; ++c) {
                    double best = 0.0;
                    int64_t bi = -1;
                    for (int64_t r = 0; r < k; ++r)
                        for (int64_t t = 0; t < k; ++t) {
                            const int64_t h = pp * s - p + r, w = qq * s - p + t;
                            if (h < 0 || h >= H || w < 0 || w >= W) continue;
                            const int64_t idx = ((n * H + h) * W + w) * C + c;
                            if (bi < 0 || x[idx] > best) {
                                best = x[idx];
                                bi = idx;
                            }
                        }
                    const int64_t o = ((n * P + pp) * Q + qq) * C + c;
                    y[o] = bi < 0 ? 0.0 : best;
                    if (arg) arg[o] = bi;
                }
    return ORC_OK;
}

/* Gradient of max pooling: each output gradient goes to the input its window selected. */
int orc_maxpool_bwd(const int32_t* dims, const double* dy, const int64_t* arg, double* dx) {
    const int64_t N = dims[0], H = dims[1], W = dims[2], C = dims[3], k = dims[4], s = dims[5],
                  p = dims[6];
    const int64_t P = (H + 2 * p - k) / s + 1, Q = (W + 2 * p - k) / s + 1;
    for (int64_t i = 0; i < N * H * W * C; ++i) dx[i] = 0.0;
    for (int64_t o = 0; o < N * P * Q * C; ++o)
        if (arg[o] >= 0) dx[arg[o]] += dy[o];
    return ORC_OK;
}

/* Global average pooling: y[n][c] = mean over (h, w) of x[n][h][w][c]. */
void orc_avgpool_global(const int32_t* dims /* N,H,W,C */, const double* x, double* y) {
    const int64_t N = dims[0], HW = (int64_t)dims[1] * dims[2], C = dims[3];
    for (int64_t n = 0; n < N; ++n)
        for (int64_t c = 0; c < C; ++c) {
            double acc = 0.0;
            for (int64_t i = 0; i < HW; ++i) acc += x[(n * HW + i) * C + c];
            y[n * C + c] = acc / (double)HW;
        }
}

/* Batch normalisation, inference form: y = gamma (x - mean) / sqrt(var + eps) + beta. */
void orc_bn_infer(const double* x, int64_t rows, int64_t C, const double* gamma, const double* beta,
                  const double* mean, const double* var, double eps, double* y) {
    for (int64_t i = 0; i < rows; ++i)
        for (int64_t c = 0; c < C; ++c)
            y[i * C + c] = gamma[c] * (x[i * C + c] - mean[c]) / sqrt(var[c] + eps) + beta[c];
}

/* Batch normalisation, training form: per-channel mean and biased variance over the
 * `rows` = N*H*W positions, y = gamma * (x - mean) / sqrt(var + eps) + beta. */
void orc_bn_train_fwd(const double* x, int64_t rows, int64_t C, const double* gamma,
                      const double* beta, double eps, double* y, double* mean_out,
                      double* var_out) {
    for (int64_t c = 0; c < C; ++c) {
        double m = 0.0;
        for (int64_t i = 0; i < rows; ++i) m += x[i * C + c];
        m /= (double)rows;
        double v = 0.0;
        for (int64_t i = 0; i < rows; ++i) v += (x[i * C + c] - m) * (x[i * C + c] - m);
        v /= (double)rows;
        const double inv = 1.0 / sqrt(v + eps);
        for (int64_t i = 0; i < rows; ++i) y[i * C + c] = gamma[c] * (x[i * C + c] - m) * inv + beta[c];
        if (mean_out) mean_out[c] = m;
        if (var_out) var_out[c] = v;
    }
}

/* Gradient of the training form of batch normalisation (chain rule through the batch
 * mean and variance):  dx = gamma / sqrt(var + eps) * (dy - mean(dy) - xhat mean(dy xhat)),
 * dgamma = sum dy xhat, dbeta = sum dy. */
void orc_bn_train_bwd(const double* x, const double* dy, int64_t rows, int64_t C,
                      const double* gamma, double eps, double* dx, double* dgamma, double* dbeta) {
    for (int64_t c = 0; c < C; ++c) {
        double m = 0.0;
        for (int64_t i = 0; i < rows; ++i) m += x[i * C + c];
        m /= (double)rows;
        double v = 0.0;
        for (int64_t i = 0; i < rows; ++i) v += (x[i * C + c] - m) * (x[i * C + c] - m);
        v /= (double)rows;
        const double inv = 1.0 / sqrt(v + eps);
        double sdy = 0.0, sdyx = 0.0;
        for (int64_t i = 0; i < rows; ++i) {
            const double xh = (x[i * C + c] - m) * inv;
            sdy += dy[i * C + c];
            sdyx += dy[i * C + c] * xh;
        }
        for (int64_t i = 0; i < rows; ++i) {
            const double xh = (x[i * C + c] - m) * inv;
            dx[i * C + c] = gamma[c] * inv * (dy[i * C + c] - sdy / rows - xh * sdyx / rows);
        }
        if (dgamma) dgamma[c] = sdyx;
        if (dbeta) dbeta[c] = sdy;
    }
}

/* Softmax cross-entropy, mean over the batch: loss = mean_n (logsumexp(z_n) - z_n[y_n]);
 * dz[n][j] = (softmax(z_n)[j] - [j == y_n]) / N. */
double orc_softmax_xent(const double* z, const int64_t* labels, int64_t N, int64_t classes,
                        double* dz) {
    double loss = 0.0;
    for (int64_t n = 0; n < N; ++n) {
        const double* zn = z + n * classes;
        double mx = zn[0];
        for (int64_t j = 1; j < classes; ++j)
            if (zn[j] > mx) mx = zn[j];
        double se = 0.0;
        for (int64_t j = 0; j < classes; ++j) se += exp(zn[j] - mx);
        const double lse = mx + log(se);
        loss += lse - zn[labels[n]];
        if (dz)
            for (int64_t j = 0; j < classes; ++j)
                dz[n * classes + j] = (exp(zn[j] - lse) - (j == labels[n] ? 1.0 : 0.0)) / (double)N;
    }
    return loss / (double)N;
}

/* Threads of the parallel loops (timing only: every routine gives the same result for any
 * thread count, each output element being computed by one thread in a fixed order). */
#ifdef _OPENMP
#include <omp.h>
void orc_set_threads(int n) {
    if (n >= 1) omp_set_num_threads(n);
}
int orc_max_threads(void) { return omp_get_max_threads(); }
#else
void orc_set_threads(int n) { (void)n; }
int orc_max_threads(void) { return 1; }
#endif
