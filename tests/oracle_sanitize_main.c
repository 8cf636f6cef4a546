/*
 * Driver for running the oracle under AddressSanitizer and UndefinedBehaviorSanitizer
 * (built and run by tests/test_oracle_sanitize.py).  Every oracle routine is called on small
 * layers whose buffers are allocated to exactly the documented sizes, so an out-of-bounds
 * access, a use of uninitialised heap memory through an overflow, or undefined arithmetic
 * aborts the program.  Exit status 0 = every call returned success.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

void orc_round_bf16(const float* in, int64_t count, double* out);
void orc_codes_of_bits(uint64_t start, int64_t count, int8_t* codes);
int orc_quantize(const float* w, int64_t K, int64_t n, int8_t* codes, double* alpha64, float* alpha32,
                 int64_t* b1_size, int64_t* b2_size, double* b1_sum, double* b2_sum);
int orc_quantize_variant(const float* w, int64_t K, int64_t n, float t, const float* uniform, int8_t* codes,
                         double* alpha64, float* alpha32, int64_t* b1_size, int64_t* b2_size);
int64_t orc_packed_words(int64_t K, int64_t n);
int orc_pack(const int8_t* codes, int64_t K, int64_t n, uint32_t* words);
int orc_unpack(const uint32_t* words, int64_t K, int64_t n, int8_t* codes);
int orc_out_dims(const int32_t* d, int32_t* P, int32_t* Q);
int orc_conv_fwd(const int32_t* d, const double* x, const int8_t* codes, const double* alpha, int form, double* y);
int orc_conv_fwd_dense(const int32_t* d, const double* x, const double* wts, double* y);
void orc_quantize_act_i8(const float* x, int64_t count, float inv, int8_t* q);
int orc_conv_fwd_i8(const int32_t* d, const int8_t* xq, const int8_t* codes, const float* alpha, float s, int relu,
                    int64_t* acc_out, float* y);
int orc_conv_bwd_data(const int32_t* d, const double* dy, const int8_t* codes, const double* alpha, double* dx);
int orc_conv_bwd_weight(const int32_t* d, const double* x, const double* dy, double* dw);
int orc_conv_fwd_sampled_bf16(const int32_t* d, const uint16_t* x, const int8_t* codes, const double* alpha,
                              const int64_t* idx, int64_t count, double* out);
int orc_conv_bwd_data_sampled_bf16(const int32_t* d, const uint16_t* dy, const int8_t* codes, const double* alpha,
                                   const int64_t* idx, int64_t count, double* out);
int orc_conv_bwd_weight_sampled_bf16(const int32_t* d, const uint16_t* x, const uint16_t* dy, const int64_t* idx,
                                     int64_t count, double* out);
void orc_sgd(double* w, double* v, const double* g, int64_t count, double eta, double mu, double lambda);
void orc_sgd_f32(float* w, float* v, const float* g, int64_t count, float eta, float mu, float lambda);
int orc_maxpool_fwd(const int32_t* dims, const double* x, double* y, int64_t* arg);
int orc_maxpool_bwd(const int32_t* dims, const double* dy, const int64_t* arg, double* dx);
void orc_avgpool_global(const int32_t* dims, const double* x, double* y);
void orc_bn_infer(const double* x, int64_t rows, int64_t C, const double* gamma, const double* beta,
                  const double* mean, const double* var, double eps, double* y);
void orc_bn_train_fwd(const double* x, int64_t rows, int64_t C, const double* gamma, const double* beta, double eps,
                      double* y, double* mean_out, double* var_out);
void orc_bn_train_bwd(const double* x, const double* dy, int64_t rows, int64_t C, const double* gamma, double eps,
                      double* dx, double* dgamma, double* dbeta);
double orc_softmax_xent(const double* z, const int64_t* labels, int64_t N, int64_t classes, double* dz);

static uint64_t state = 88172645463325252ull;
static double urand(void) { /* xorshift64, in [0, 1) */
    state ^= state << 13;
    state ^= state >> 7;
    state ^= state << 17;
    return (double)(state >> 11) / 9007199254740992.0;
}
#define NEW(T, n) ((T*)calloc((size_t)(n) > 0 ? (size_t)(n) : 1, sizeof(T)))

static int fails = 0;
#define CHECK(call)                                          \
    do {                                                     \
        if ((call) != 0) {                                   \
            fprintf(stderr, "failed: %s\n", #call);          \
            ++fails;                                         \
        }                                                    \
    } while (0)

static void layer(int n, int h, int w, int c, int k, int r, int s, int st, int pd) {
    const int32_t d[11] = {n, h, w, c, k, r, s, st, st, pd, pd};
    int32_t P, Q;
    CHECK(orc_out_dims(d, &P, &Q));
    const int64_t nx = (int64_t)n * h * w * c, ny = (int64_t)n * P * Q * k, nf = (int64_t)r * s * c;
    float* wr = NEW(float, k * nf);
    double* x = NEW(double, nx);
    double* dy = NEW(double, ny);
    uint16_t* xb = NEW(uint16_t, nx);
    uint16_t* dyb = NEW(uint16_t, ny);
    for (int64_t i = 0; i < k * nf; ++i) wr[i] = (float)(4.0 * urand() - 2.0);
    for (int64_t i = 0; i < nx; ++i) x[i] = 2.0 * urand() - 1.0, xb[i] = (uint16_t)(0x3F00 + (i & 0x7F));
    for (int64_t i = 0; i < ny; ++i) dy[i] = 2.0 * urand() - 1.0, dyb[i] = (uint16_t)(0xBF00 + (i & 0x7F));
    int8_t* codes = NEW(int8_t, k * nf);
    int8_t* codes2 = NEW(int8_t, k * nf);
    double* a64 = NEW(double, k);
    float* a32 = NEW(float, k);
    int64_t *b1 = NEW(int64_t, k), *b2 = NEW(int64_t, k);
    double *s1 = NEW(double, k), *s2 = NEW(double, k);
    CHECK(orc_quantize(wr, k, nf, codes, a64, a32, b1, b2, s1, s2));
    float* uni = NEW(float, k * nf);
    for (int64_t i = 0; i < k * nf; ++i) uni[i] = (float)urand();
    CHECK(orc_quantize_variant(wr, k, nf, 0.5f, NULL, codes2, a64, a32, b1, b2));
    CHECK(orc_quantize_variant(wr, k, nf, 1.0f, uni, codes2, a64, a32, b1, b2));
    uint32_t* words = NEW(uint32_t, orc_packed_words(k, nf));
    CHECK(orc_pack(codes, k, nf, words));
    CHECK(orc_unpack(words, k, nf, codes2));
    double* y = NEW(double, ny);
    for (int form = 0; form < 3; ++form) CHECK(orc_conv_fwd(d, x, codes, a64, form, y));
    double* wd = NEW(double, k * nf);
    for (int64_t i = 0; i < k * nf; ++i) wd[i] = wr[i];
    CHECK(orc_conv_fwd_dense(d, x, wd, y));
    double* dx = NEW(double, nx);
    double* dw = NEW(double, k * nf);
    if (st == 1) CHECK(orc_conv_bwd_data(d, dy, codes, a64, dx));
    CHECK(orc_conv_bwd_weight(d, x, dy, dw));
    int64_t idx[3] = {0, ny / 2, ny - 1}, idxx[3] = {0, nx / 2, nx - 1}, idxw[3] = {0, k * nf / 2, k * nf - 1};
    double out[3];
    CHECK(orc_conv_fwd_sampled_bf16(d, xb, codes, a64, idx, 3, out));
    if (st == 1) CHECK(orc_conv_bwd_data_sampled_bf16(d, dyb, codes, a64, idxx, 3, out));
    CHECK(orc_conv_bwd_weight_sampled_bf16(d, xb, dyb, idxw, 3, out));
    float* xf = NEW(float, nx);
    int8_t* xq = NEW(int8_t, nx);
    for (int64_t i = 0; i < nx; ++i) xf[i] = (float)(300.0 * urand() - 150.0);
    orc_quantize_act_i8(xf, nx, 0.9f, xq);
    int64_t* acc = NEW(int64_t, ny);
    float* yf = NEW(float, ny);
    CHECK(orc_conv_fwd_i8(d, xq, codes, a32, 0.01f, 1, acc, yf));
    double* rb = NEW(double, nx);
    orc_round_bf16(xf, nx, rb);
    free(wr); free(x); free(dy); free(xb); free(dyb); free(codes); free(codes2); free(a64); free(a32);
    free(b1); free(b2); free(s1); free(s2); free(uni); free(words); free(y); free(wd); free(dx); free(dw);
    free(xf); free(xq); free(acc); free(yf); free(rb);
}

static void glue(void) {
    const int N = 2, H = 7, W = 5, C = 3;
    const int32_t pd[7] = {N, H, W, C, 3, 2, 1};
    const int P = (H + 2 - 3) / 2 + 1, Q = (W + 2 - 3) / 2 + 1;
    double* x = NEW(double, N * H * W * C);
    for (int i = 0; i < N * H * W * C; ++i) x[i] = urand();
    double* y = NEW(double, N * P * Q * C);
    int64_t* arg = NEW(int64_t, N * P * Q * C);
    double* dx = NEW(double, N * H * W * C);
    CHECK(orc_maxpool_fwd(pd, x, y, arg));
    CHECK(orc_maxpool_bwd(pd, y, arg, dx));
    const int32_t ad[4] = {N, H, W, C};
    double* g = NEW(double, N * C);
    orc_avgpool_global(ad, x, g);
    const int64_t rows = N * H * W;
    double *gm = NEW(double, C), *bt = NEW(double, C), *mu = NEW(double, C), *var = NEW(double, C);
    for (int c = 0; c < C; ++c) gm[c] = 1.0, bt[c] = 0.1, mu[c] = 0.0, var[c] = 1.0;
    double* bn = NEW(double, rows * C);
    orc_bn_infer(x, rows, C, gm, bt, mu, var, 1e-5, bn);
    orc_bn_train_fwd(x, rows, C, gm, bt, 1e-5, bn, mu, var);
    double *dg = NEW(double, C), *db = NEW(double, C);
    orc_bn_train_bwd(x, x, rows, C, gm, 1e-5, dx, dg, db);
    int64_t labels[2] = {0, 2};
    double dz[6];
    (void)orc_softmax_xent(x, labels, 2, 3, dz);
    double w[5] = {1, 2, 3, 4, 5}, v[5] = {0}, gr[5] = {1, 1, 1, 1, 1};
    orc_sgd(w, v, gr, 5, 0.1, 0.9, 1e-4);
    float wf[5] = {1, 2, 3, 4, 5}, vf[5] = {0}, gf[5] = {1, 1, 1, 1, 1};
    orc_sgd_f32(wf, vf, gf, 5, 0.1f, 0.9f, 1e-4f);
    int8_t cb[4096];
    orc_codes_of_bits(0xFFFFF800ull, 4096, cb); /* wraps past 2^32 */
    free(x); free(y); free(arg); free(dx); free(g); free(gm); free(bt); free(mu); free(var); free(bn);
    free(dg); free(db);
}

int main(void) {
    layer(1, 1, 1, 1, 1, 1, 1, 1, 0);
    layer(2, 7, 6, 3, 5, 3, 3, 1, 1);
    layer(1, 9, 8, 8, 70, 5, 3, 2, 2);
    layer(2, 5, 4, 16, 65, 1, 1, 1, 3);
    layer(1, 6, 6, 5, 9, 6, 6, 1, 0);
    glue();
    if (fails) fprintf(stderr, "%d oracle calls failed\n", fails);
    return fails ? 1 : 0;
}
