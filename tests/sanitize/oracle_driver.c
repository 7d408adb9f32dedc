/* Drives the oracle's functions on small random inputs of several shapes
 * (ragged sizes, padded transforms, transposed convolutions, every Hadamard
 * order family) for a build under AddressSanitizer and UndefinedBehavior-
 * Sanitizer; exits 0 when every call returns its success status. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

int orc_sylvester(int b, int8_t *H);
int orc_paley(int q, int kind, int8_t *H);
int orc_hadamard(int m, int8_t *H);
int orc_order(int C, int mmax);
int orc_activation_transform(const float *x, int64_t P, int C, int b, float *S);
void orc_quantize_symmetric(const float *S, int64_t nsamp, int64_t per, int8_t *q, float *scale);
void orc_quantize_affine(const float *S, int64_t nsamp, int64_t per, int8_t *q, float *scale, int32_t *zero);
int orc_prepare_weights(int cin, int cout, int k, int transposed, int hblock, int form, const float *w,
                        const float *bias, int8_t *wq, float *w_scale, float *w_bias, float *w_real);
int orc_out_size(int in, int k, int stride, int pad, int transposed, int out_pad);
void orc_conv_int8(const int8_t *xq, const int32_t *zx, int n, int h, int w, int cin_p, const int8_t *wq,
                   int cout_p, int k, int stride, int pad, int transposed, int out_pad, int32_t *acc);
void orc_conv_f64(const double *x, int n, int h, int w, int cin, const double *wf, int cout, int k, int stride,
                  int pad, int transposed, int out_pad, double *y);
int orc_epilogue(const int32_t *acc, int n, int64_t pix, int cout, int cout_p, int form, int hblock,
                 const float *sx, const float *sw, const float *bias, float *y);
void orc_wh_z(const int32_t *acc, int n, int64_t pix, int cout_p, const float *sx, const float *sw,
              const float *bias, float *z);
int orc_int_requant_params(int cout_p, float s_x, const float *s_w, const float *bias, float s_y, int beta_in,
                           int beta_out, int K, int gain, int32_t *M, int32_t *b_int);
int orc_int_transition(const int32_t *acc, int64_t P, int cout, int cout_p, const int32_t *M, const int32_t *b_int,
                       int n, int wb, int nb, int8_t *q);
int orc_range_expansion(const float *x, int n, int64_t P, int C, int b, float *ax, float *ah, int32_t *flags);

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static double urand(void)
{
    rng_state ^= rng_state << 13;
    rng_state ^= rng_state >> 7;
    rng_state ^= rng_state << 17;
    return (double)(rng_state >> 11) / 9007199254740992.0;
}
static float *frand(size_t n, float scale)
{
    float *p = malloc(n * sizeof(float));
    for (size_t i = 0; i < n; ++i) p[i] = (float)((urand() * 2 - 1) * scale);
    return p;
}

#define CHECK(c) do { if (!(c)) { fprintf(stderr, "failed: %s (line %d)\n", #c, __LINE__); return 1; } } while (0)

static int layer(int n, int h, int w, int cin, int cout, int k, int stride, int pad, int tr, int op, int form, int hb)
{
    const int cin_p = form == 0 ? (cin + hb - 1) / hb * hb : cin;
    const int cout_p = form == 1 ? (cout + hb - 1) / hb * hb : cout;
    float *x = frand((size_t)n * h * w * cin, 3.0f);
    float *S = malloc(sizeof(float) * (size_t)n * h * w * cin_p);
    CHECK(orc_activation_transform(x, (int64_t)n * h * w, cin, form == 0 ? hb : 1, S) == 0);
    int8_t *xq = malloc((size_t)n * h * w * cin_p);
    float *sx = malloc(sizeof(float) * n);
    orc_quantize_symmetric(S, n, (int64_t)h * w * cin_p, xq, sx);
    int32_t *zx = malloc(sizeof(int32_t) * n);
    orc_quantize_affine(S, n, (int64_t)h * w * cin_p, xq, sx, zx);
    orc_quantize_symmetric(S, n, (int64_t)h * w * cin_p, xq, sx);
    float *wt = frand((size_t)cout * cin * k * k, 0.05f), *b = frand(cout, 0.05f);
    int8_t *wq = malloc((size_t)cout_p * k * k * cin_p);
    float *ws = malloc(sizeof(float) * cout_p), *wb = malloc(sizeof(float) * cout_p);
    float *wr = malloc(sizeof(float) * (size_t)cout_p * k * k * cin_p);
    CHECK(orc_prepare_weights(cin, cout, k, tr, hb, form, wt, b, wq, ws, wb, wr) == 0);
    const int ho = orc_out_size(h, k, stride, pad, tr, op), wo = orc_out_size(w, k, stride, pad, tr, op);
    CHECK(ho > 0 && wo > 0);
    const int64_t P = (int64_t)ho * wo;
    int32_t *acc = malloc(sizeof(int32_t) * (size_t)n * P * cout_p);
    orc_conv_int8(xq, NULL, n, h, w, cin_p, wq, cout_p, k, stride, pad, tr, op, acc);
    orc_conv_int8(xq, zx, n, h, w, cin_p, wq, cout_p, k, stride, pad, tr, op, acc);
    float *y = malloc(sizeof(float) * (size_t)n * P * cout);
    CHECK(orc_epilogue(acc, n, P, cout, cout_p, form, hb, sx, ws, wb, y) == 0);
    if (form == 1) {
        float *z = malloc(sizeof(float) * (size_t)n * P * cout_p);
        orc_wh_z(acc, n, P, cout_p, sx, ws, wb, z);
        free(z);
    }
    int32_t *M = malloc(sizeof(int32_t) * cout_p), *bi = malloc(sizeof(int32_t) * cout_p);
    int8_t *q = malloc((size_t)n * P * cout);
    if ((hb & (hb - 1)) == 0) {   /* the integer transition takes Sylvester blocks */
        const int sh = orc_int_requant_params(cout_p, sx[0], ws, wb, 0.05f, form == 0 ? hb : 1,
                                              form == 1 ? hb : 1, k * k * cin_p, form == 1 ? hb : 1, M, bi);
        CHECK(sh >= 0);
        CHECK(orc_int_transition(acc, (int64_t)n * P, cout, cout_p, M, bi, sh, form == 1 ? hb : 1, 1, q) == 0);
    }
    float *ax = malloc(sizeof(float) * n), *ah = malloc(sizeof(float) * n);
    int32_t *fl = malloc(sizeof(int32_t) * n);
    if ((hb & (hb - 1)) == 0) CHECK(orc_range_expansion(x, n, (int64_t)h * w, cin, hb, ax, ah, fl) == 0);
    double *xd = malloc(sizeof(double) * (size_t)n * h * w * cin), *wd = malloc(sizeof(double) * (size_t)cout * k * k * cin);
    for (size_t i = 0; i < (size_t)n * h * w * cin; ++i) xd[i] = x[i];
    for (size_t i = 0; i < (size_t)cout * k * k * cin; ++i) wd[i] = 0.01 * (double)(i % 7);
    double *yd = malloc(sizeof(double) * (size_t)n * P * cout);
    orc_conv_f64(xd, n, h, w, cin, wd, cout, k, stride, pad, tr, op, yd);
    free(x); free(S); free(xq); free(sx); free(zx); free(wt); free(b); free(wq); free(ws); free(wb); free(wr);
    free(acc); free(y); free(M); free(bi); free(q); free(ax); free(ah); free(fl); free(xd); free(wd); free(yd);
    return 0;
}

int main(void)
{
    int8_t *H = malloc(400 * 400);
    for (int b = 1; b <= 128; b *= 2) CHECK(orc_sylvester(b, H) == 0);
    CHECK(orc_paley(27, 1, H) == 0 && orc_paley(25, 2, H) == 0 && orc_paley(11, 1, H) == 0);
    for (int m = 1; m <= 400; ++m) orc_hadamard(m, H);
    for (int C = 1; C < 300; ++C) CHECK(orc_order(C, 4096) > 0);
    free(H);
    CHECK(layer(2, 9, 11, 192, 192, 5, 2, 2, 0, 0, 0, 64) == 0);
    CHECK(layer(1, 8, 7, 192, 320, 5, 2, 2, 0, 0, 1, 64) == 0);
    CHECK(layer(2, 7, 9, 3, 192, 5, 2, 2, 0, 0, 1, 64) == 0);
    CHECK(layer(1, 5, 6, 192, 192, 5, 2, 2, 1, 1, 0, 64) == 0);
    CHECK(layer(1, 6, 5, 128, 128, 1, 1, 0, 0, 0, 0, 128) == 0);
    CHECK(layer(1, 5, 5, 17, 24, 3, 1, 1, 0, 0, 0, 20) == 0);
    CHECK(layer(1, 4, 4, 40, 50, 3, 2, 1, 0, 0, 1, 52) == 0);
    printf("oracle driver ok\n");
    return 0;
}
