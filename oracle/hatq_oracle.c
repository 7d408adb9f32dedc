/*
 * CPU oracle for the Hadamard-domain INT8 linear operator (HaTQ).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or call
 * this file; only the tests, the smoke check and the benchmark's CPU-baseline leg
 * do.  It shares no code, header, table or helper with the HIP library: every
 * step is re-derived here from the paper in the plainest form available
 * (dense matrices, direct loops, fp64 sums, IEEE fp32 division, RNE rounding).
 *
 * Notation (paper): Y = X W^T + b (Eq. supp_linear_operator); a Sylvester matrix
 * H~_m with H~ H~^T = m I (Eq. supp_hadamard_properties, Eq. supp_sylvester);
 * symmetric quantizer with q_max = 127 and s = ||x||_inf / 127 (Eq. symmetric_q,
 * Eq. current_scale); INT32 accumulation (Eq. integer_accumulation); accumulator
 * scale s_x s_w,c (Eq. accumulator_scale); DH and WH forms (Eq.
 * double_hadamard_quantization, Eq. weight_only_hadamard_quantization, and their
 * padded versions Eq. supp_padded_dh, Eq. supp_padded_wh).
 *
 * Readings taken where the paper is silent (each listed in the design notes):
 *  - round() is IEEE round-half-to-even; x/s is an IEEE fp32 division.
 *  - The transform is the block-diagonal B_C = I_{C_pad/b} (x) H~_b, unnormalized;
 *    the 1/sqrt(b) normalizations of both sides are absorbed into the dequant
 *    scale as one exact factor 1/b (Sec. IV-B "absorbed into fixed-point
 *    requantization"; Supplementary "Deployment Realization").
 *  - One activation scale per sample (per input tensor at inference).
 *  - An all-zero tensor or weight row gets scale 1 and all-zero codes.
 *  - Bias is added in fp32 after dequantization, in the accumulator basis
 *    (transformed for WH, Eq. supp_padded_wh_parameters), before the WH
 *    output-basis restore; per-channel scales are applied before that restore
 *    (Supplementary "General Nonlinearities", ordering rule).
 *
 * Built with -O2 -fopenmp -ffp-contract=off (no fast-math): every fp32 product
 * and quotient below is a single correctly rounded IEEE operation.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* Thread count of the OpenMP loops below (timing of the oracle as a CPU     */
/* baseline; results do not depend on it: every parallel loop writes disjoint */
/* outputs and reduces only with max).  Returns the count now in effect.      */
int orc_set_threads(int n)
{
    if (n > 0) omp_set_num_threads(n);
    return omp_get_max_threads();
}

static int is_pow2(int b) { return b >= 1 && (b & (b - 1)) == 0; }
static int round_up(int v, int m) { return (v + m - 1) / m * m; }

/* ------------------------------------------------------------------------- */
/* O1. Sylvester matrix by its recursion (Eq. supp_sylvester):                */
/*     H~_1 = [1],  H~_2m = [[H~_m, H~_m], [H~_m, -H~_m]].                   */
/* H is b*b, row-major.  Returns 0, or -1 when b is not a power of two.       */
/* ------------------------------------------------------------------------- */
int orc_sylvester(int b, int8_t *H)
{
    if (!is_pow2(b)) return -1;
    H[0] = 1;
    for (int m = 1; m < b; m *= 2)
        for (int i = 0; i < m; ++i)
            for (int j = 0; j < m; ++j) {
                int8_t v = H[i * b + j];
                H[i * b + (j + m)] = v;
                H[(i + m) * b + j] = v;
                H[(i + m) * b + (j + m)] = (int8_t)-v;
            }
    return 0;
}

/* Paley constructions (supplementary, Hadamard construction), for an odd    */
/* prime power q = p^k.  chi is the quadratic character of the finite field   */
/* F_q (chi(0) = 0, chi(a) = 1 for a nonzero square, -1 otherwise) and Q the  */
/* Jacobsthal matrix Q[i][j] = chi(x_j - x_i) over the field elements x_i.    */
/*  Paley-I  (q = 3 mod 4, order q + 1): H = I + [[0, 1^T], [-1, Q]].         */
/*  Paley-II (q = 1 mod 4, order 2(q + 1)): with the symmetric conference     */
/*           matrix C = [[0, 1^T], [1, Q]], every entry C[i][j] becomes the   */
/*           2x2 block [[1, -1], [-1, -1]] where C[i][j] = 0 and              */
/*           C[i][j] * [[1, 1], [1, -1]] otherwise.                           */
/* Field elements: x_e for e = 0 .. q-1 is the polynomial sum_i d_i t^i with  */
/* e = sum_i d_i p^i (0 <= d_i < p), arithmetic modulo p and modulo the       */
/* smallest monic irreducible polynomial of degree k over F_p (smallest by    */
/* its lower coefficients read as the base-p number sum_i f_i p^i).  For k = 1 */
/* this is the integers modulo p.  Returns 0, or -1 if q is not such a power. */
#define GF_MAXK 16

/* q = p^k with p prime and k >= 1: returns 1 and sets p, k. */
static int prime_power(int q, int *p, int *k)
{
    if (q < 2) return 0;
    int d = 2;
    while (q % d) ++d;              /* the smallest prime factor */
    int e = 0, r = q;
    while (r % d == 0) { r /= d; ++e; }
    if (r != 1) return 0;
    *p = d;
    *k = e;
    return 1;
}

typedef struct {
    int p, k, q;
    int f[GF_MAXK + 1];             /* monic modulus, f[k] = 1 */
} gf_t;

static void gf_digits(const gf_t *F, int e, int *d)
{
    for (int i = 0; i < F->k; ++i) { d[i] = e % F->p; e /= F->p; }
}

static int gf_pack(const gf_t *F, const int *d)
{
    int e = 0;
    for (int i = F->k - 1; i >= 0; --i) e = e * F->p + d[i];
    return e;
}

static int gf_sub(const gf_t *F, int a, int b)
{
    int da[GF_MAXK], db[GF_MAXK];
    gf_digits(F, a, da);
    gf_digits(F, b, db);
    for (int i = 0; i < F->k; ++i) da[i] = ((da[i] - db[i]) % F->p + F->p) % F->p;
    return gf_pack(F, da);
}

static int gf_mul(const gf_t *F, int a, int b)
{
    const int p = F->p, k = F->k;
    int da[GF_MAXK], db[GF_MAXK], c[2 * GF_MAXK] = {0};
    gf_digits(F, a, da);
    gf_digits(F, b, db);
    for (int i = 0; i < k; ++i)
        for (int j = 0; j < k; ++j) c[i + j] = (c[i + j] + da[i] * db[j]) % p;
    /* t^d = t^(d-k) * t^k and t^k = -(f_0 + ... + f_(k-1) t^(k-1)) */
    for (int d = 2 * k - 2; d >= k; --d) {
        const int v = c[d];
        c[d] = 0;
        for (int i = 0; i < k; ++i) c[d - k + i] = ((c[d - k + i] - v * F->f[i]) % p + p) % p;
    }
    return gf_pack(F, c);
}

/* Whether the monic g of degree dg divides the monic f of degree k over F_p. */
static int poly_divides(const int *g, int dg, const int *f, int k, int p)
{
    int r[GF_MAXK + 1];
    for (int i = 0; i <= k; ++i) r[i] = f[i];
    for (int d = k; d >= dg; --d) {
        const int v = r[d];
        if (!v) continue;
        for (int i = 0; i <= dg; ++i) r[d - dg + i] = ((r[d - dg + i] - v * g[i]) % p + p) % p;
    }
    for (int i = 0; i < dg; ++i)
        if (r[i]) return 0;
    return 1;
}

/* Irreducible: no monic divisor of degree 1 .. k/2. */
static int poly_irreducible(const int *f, int k, int p)
{
    int g[GF_MAXK + 1];
    for (int dg = 1; 2 * dg <= k; ++dg) {
        int count = 1;
        for (int i = 0; i < dg; ++i) count *= p;
        for (int c = 0; c < count; ++c) {
            int v = c;
            for (int i = 0; i < dg; ++i) { g[i] = v % p; v /= p; }
            g[dg] = 1;
            if (poly_divides(g, dg, f, k, p)) return 0;
        }
    }
    return 1;
}

static int gf_init(gf_t *F, int q)
{
    int p, k;
    if (!prime_power(q, &p, &k) || k > GF_MAXK) return -1;
    F->p = p;
    F->k = k;
    F->q = q;
    for (int c = 0; c < q; ++c) {   /* lower coefficients as a base-p number, ascending */
        int v = c;
        for (int i = 0; i < k; ++i) { F->f[i] = v % p; v /= p; }
        F->f[k] = 1;
        if (poly_irreducible(F->f, k, p)) return 0;
    }
    return -1;
}

/* chi[e] for every element e of F_q, from the set of squares. */
static int *gf_quadratic_character(const gf_t *F)
{
    int *chi = (int *)malloc(sizeof(int) * (size_t)F->q);
    for (int e = 0; e < F->q; ++e) chi[e] = -1;
    for (int x = 1; x < F->q; ++x) chi[gf_mul(F, x, x)] = 1;
    chi[0] = 0;
    return chi;
}

/* q is an odd prime power of the residue the Paley kind needs. */
static int paley_q_ok(int q, int kind)
{
    int p, k;
    if (q < 3 || q % 2 == 0 || !prime_power(q, &p, &k)) return 0;
    return kind == 1 ? q % 4 == 3 : kind == 2 ? q % 4 == 1 : 0;
}

int orc_paley(int q, int kind, int8_t *H)
{
    if (!paley_q_ok(q, kind)) return -1;
    gf_t F;
    if (gf_init(&F, q)) return -1;
    int *chi = gf_quadratic_character(&F);
    const int n = q + 1;
    /* matrix index i >= 1 stands for the field element x_(i-1) */
    if (kind == 1) {
        for (int i = 0; i < n; ++i)
            for (int j = 0; j < n; ++j) {
                int s;
                if (i == 0) s = j == 0 ? 0 : 1;
                else if (j == 0) s = -1;
                else s = chi[gf_sub(&F, j - 1, i - 1)];
                H[i * n + j] = (int8_t)((i == j ? 1 : 0) + s);
            }
    } else {
        const int m = 2 * n;
        for (int i = 0; i < n; ++i)
            for (int j = 0; j < n; ++j) {
                int c;
                if (i == 0 || j == 0) c = (i == j) ? 0 : 1;
                else c = chi[gf_sub(&F, j - 1, i - 1)];
                for (int a = 0; a < 2; ++a)
                    for (int b = 0; b < 2; ++b) {
                        int v;
                        if (c == 0) v = (a == 0 && b == 0) ? 1 : -1;
                        else v = (a == 1 && b == 1) ? -c : c;
                        H[(2 * i + a) * m + 2 * j + b] = (int8_t)v;
                    }
            }
    }
    free(chi);
    return 0;
}

/* The supported set M_H: the Sylvester orders, the Paley orders, and         */
/* Kronecker products of supported orders.  The construction of order m:     */
/*  (1) if m = b * 2^j with b = 1 or a Paley order: P_b (x) H~_(m/b) for the   */
/*      smallest such b (Paley-I preferred over Paley-II for the same b);     */
/*  (2) else, if m = a * c with a and c supported, 1 < a <= c: H_a (x) H_c    */
/*      for the smallest such a, each factor by this rule.                    */
/* orc_hadamard_base returns the b of form (1) with its construction (kind 0: */
/* b = 1, else the Paley kind and q), or -1 when m has no form (1).           */
int orc_hadamard_base(int m, int *kind, int *q)
{
    if (m < 1) return -1;
    for (int b = 1; b <= m; ++b) {
        if (m % b || !is_pow2(m / b)) continue;
        if (b == 1) { *kind = 0; *q = 0; return 1; }
        if (paley_q_ok(b - 1, 1)) { *kind = 1; *q = b - 1; return b; }
        if (b % 2 == 0 && paley_q_ok(b / 2 - 1, 2)) { *kind = 2; *q = b / 2 - 1; return b; }
    }
    return -1;
}

static int supported(int m);

/* The smallest a of form (2), or -1. */
int orc_hadamard_split(int m)
{
    int kind, q;
    if (m < 1 || orc_hadamard_base(m, &kind, &q) > 0) return -1;
    for (int a = 2; a * a <= m; ++a)
        if (m % a == 0 && supported(a) && supported(m / a)) return a;
    return -1;
}

static int supported(int m)
{
    int kind, q;
    return orc_hadamard_base(m, &kind, &q) > 0 || orc_hadamard_split(m) > 0;
}

/* The Hadamard matrix of order m (row-major m*m): form (1), index (a, j) ->  */
/* a * (m/b) + j; form (2), index (i, j) -> i * c + j.  -1 if unsupported.     */
int orc_hadamard(int m, int8_t *H)
{
    int kind, q;
    const int b = orc_hadamard_base(m, &kind, &q);
    int8_t *P, *S;
    int s;
    if (b > 0) {
        s = m / b;
        P = (int8_t *)malloc((size_t)b * b);
        S = (int8_t *)malloc((size_t)s * s);
        if (kind == 0) P[0] = 1;
        else orc_paley(q, kind, P);
        orc_sylvester(s, S);
    } else {
        const int a = orc_hadamard_split(m);
        if (a < 0) return -1;
        s = m / a;
        P = (int8_t *)malloc((size_t)a * a);
        S = (int8_t *)malloc((size_t)s * s);
        orc_hadamard(a, P);
        orc_hadamard(s, S);
    }
    const int pb = m / s;
    for (int a = 0; a < pb; ++a)
        for (int j = 0; j < s; ++j)
            for (int c = 0; c < pb; ++c)
                for (int l = 0; l < s; ++l)
                    H[(a * s + j) * m + c * s + l] = (int8_t)(P[a * pb + c] * S[j * s + l]);
    free(P);
    free(S);
    return 0;
}

/* Eq. hadamard_order: C_4 = 4 ceil(C / 4), m(C) = the smallest supported     */
/* order >= C_4 (searched up to mmax; -1 if none).                            */
int orc_order(int C, int mmax)
{
    if (C < 1) return -1;
    const int c4 = 4 * ((C + 3) / 4);
    for (int m = c4; m <= mmax; ++m)
        if (supported(m)) return m;
    return -1;
}

/* Dense block-diagonal transform along the last axis, fp64 in and out:       */
/*   out[r, blk*b + i] = sum_j H~_b[i][j] * in[r, blk*b + j]                   */
/* for width = nblk*b.  Summation runs over j in natural order.               */
static void block_transform_f64(const int8_t *H, int b, const double *in, double *out,
                                int64_t rows, int width)
{
    const int nblk = width / b;
    for (int64_t r = 0; r < rows; ++r)
        for (int blk = 0; blk < nblk; ++blk)
            for (int i = 0; i < b; ++i) {
                double acc = 0.0;
                for (int j = 0; j < b; ++j)
                    acc += (double)H[i * b + j] * in[r * width + blk * b + j];
                out[r * width + blk * b + i] = acc;
            }
}

/* Public wrapper: fp64 block transform of `rows` rows of width `width`. */
int orc_block_transform_f64(int b, const double *in, double *out, int64_t rows, int width)
{
    if (!supported(b) || width % b) return -1;
    int8_t *H = (int8_t *)malloc((size_t)b * b);
    orc_hadamard(b, H);
    block_transform_f64(H, b, in, out, rows, width);
    free(H);
    return 0;
}

/* ------------------------------------------------------------------------- */
/* O3. Activation operand.  DH: S = fl32(B_C x_pad) per pixel, computed in    */
/* fp64 with one rounding (Eq. input_hadamard_transform, Eq. supp_padded_     */
/* transforms: zero-pad C to C_pad = b*ceil(C/b)).  WH: b = 1, S = x.         */
/* b is any supported order (orc_hadamard), the power-of-two ones Sylvester.  */
/* x is [P, C] fp32 (P pixels), S is [P, C_pad] fp32.                         */
/* ------------------------------------------------------------------------- */
int orc_activation_transform(const float *x, int64_t P, int C, int b, float *S)
{
    if (!supported(b) || C <= 0) return -1;
    const int Cp = round_up(C, b);
    int8_t *H = (int8_t *)malloc((size_t)b * b);
    orc_hadamard(b, H);
    #pragma omp parallel
    {
        double *in = (double *)malloc(sizeof(double) * Cp);
        double *out = (double *)malloc(sizeof(double) * Cp);
        #pragma omp for schedule(static)
        for (int64_t p = 0; p < P; ++p) {
            for (int c = 0; c < Cp; ++c) in[c] = c < C ? (double)x[p * C + c] : 0.0;
            block_transform_f64(H, b, in, out, 1, Cp);
            for (int c = 0; c < Cp; ++c) S[p * Cp + c] = (float)out[c];
        }
        free(in);
        free(out);
    }
    free(H);
    return 0;
}

/* Symmetric per-tensor quantizer (Eq. symmetric_q, Eq. current_scale), one    */
/* scale per sample.  S is [nsamp, per] fp32.                                 */
/*   A = max |S|;  s = fl32(A / 127) (A > 0), else s = 1;                      */
/*   q = clamp(rne(fl32(S / s)), -127, 127).                                   */
void orc_quantize_symmetric(const float *S, int64_t nsamp, int64_t per, int8_t *q, float *scale)
{
    for (int64_t n = 0; n < nsamp; ++n) {
        const float *s_n = S + n * per;
        float A = 0.0f;
        for (int64_t i = 0; i < per; ++i) {
            float a = fabsf(s_n[i]);
            if (a > A) A = a;
        }
        const float s = A > 0.0f ? A / 127.0f : 1.0f;
        scale[n] = s;
        #pragma omp parallel for schedule(static)
        for (int64_t i = 0; i < per; ++i) {
            float t = nearbyintf(s_n[i] / s);
            if (t > 127.0f) t = 127.0f;
            if (t < -127.0f) t = -127.0f;
            q[n * per + i] = (int8_t)t;
        }
    }
}

/* Affine per-sample quantizer (Eq. uniform_q, Eq. affine_q) on the signed    */
/* 8-bit grid [q_min, q_max] = [-128, 127] (the paper's unsigned grid [0, 255]  */
/* shifted by -128: the same dequantized values, codes that a signed INT8      */
/* product takes).  With xmin' = min(min S, 0) and xmax' = max(max S, 0):       */
/*   r = fl32(xmax' - xmin');  s = fl32(r / 255) (r > 0), else s = 1, z = 0;   */
/*   z = clamp(round(q_min - xmin'/s)) = clamp(rne(fl32(-xmin' / s)) - 128)    */
/*       (q_min is an even integer, so rounding commutes with adding it);      */
/*   q = clamp(rne(fl32(S / s)) + z, -128, 127).                               */
void orc_quantize_affine(const float *S, int64_t nsamp, int64_t per, int8_t *q, float *scale, int32_t *zero)
{
    for (int64_t n = 0; n < nsamp; ++n) {
        const float *s_n = S + n * per;
        float lo = 0.0f, hi = 0.0f;
        for (int64_t i = 0; i < per; ++i) {
            if (s_n[i] < lo) lo = s_n[i];
            if (s_n[i] > hi) hi = s_n[i];
        }
        const float r = hi - lo;
        float s = 1.0f;
        int z = 0;
        if (r > 0.0f) {
            s = r / 255.0f;
            z = (int)nearbyintf(-lo / s) - 128;
            if (z < -128) z = -128;
            if (z > 127) z = 127;
        }
        scale[n] = s;
        zero[n] = z;
        #pragma omp parallel for schedule(static)
        for (int64_t i = 0; i < per; ++i) {
            float t = nearbyintf(s_n[i] / s) + (float)z;
            if (t > 127.0f) t = 127.0f;
            if (t < -128.0f) t = -128.0f;
            q[n * per + i] = (int8_t)t;
        }
    }
}

/* ------------------------------------------------------------------------- */
/* O2. Weight preparation (offline).                                          */
/* Input: PyTorch layout, OIHW [cout][cin][k][k] for a convolution, IOHW      */
/* [cin][cout][k][k] for a transposed one.  Output canonical layout OHWI:     */
/* wq[cout_pad][k][k][cin_pad], w_scale[cout_pad], w_bias[cout_pad].          */
/* The contraction index of one output is d = (kh*K + kw)*cin_pad + ci, the   */
/* Kronecker order I_{KhKw} (x) H of Eq. input_hadamard_transform.            */
/*  DH (form 0): each (co, tap) row is multiplied by B_Cin (cin padded to b); */
/*               bias untransformed.                                          */
/*  WH (form 1): each (tap, ci) column is multiplied by B_Cout (cout padded   */
/*               to b); bias b~ = B_Cout [b; 0] (Eq. supp_padded_wh_params).  */
/* Transforms in fp64 with one rounding to fp32; then per output channel      */
/* s_w = fl32(max|W'| / 127) (1 for an all-zero row) and                      */
/* wq = clamp(rne(fl32(W'/s_w)), -127, 127).  w_real (nullable) receives the  */
/* unquantized fp32 W' in the same layout.                                    */
/* ------------------------------------------------------------------------- */
int orc_prepare_weights(int cin, int cout, int k, int transposed, int hblock, int form,
                        const float *w, const float *bias,
                        int8_t *wq, float *w_scale, float *w_bias, float *w_real)
{
    if (!supported(hblock) || cin <= 0 || cout <= 0 || k <= 0 || (form != 0 && form != 1))
        return -1;
    const int cin_p = form == 0 ? round_up(cin, hblock) : cin;
    const int cout_p = form == 1 ? round_up(cout, hblock) : cout;
    const int taps = k * k;
    const int64_t per_co = (int64_t)taps * cin_p;
    double *W0 = (double *)calloc((size_t)cout_p * per_co, sizeof(double));
    float *W1 = (float *)malloc(sizeof(float) * (size_t)cout_p * per_co);
    int8_t *H = (int8_t *)malloc((size_t)hblock * hblock);
    orc_hadamard(hblock, H);

    /* canonical fp64 copy, zero padded */
    for (int co = 0; co < cout; ++co)
        for (int kh = 0; kh < k; ++kh)
            for (int kw = 0; kw < k; ++kw)
                for (int ci = 0; ci < cin; ++ci) {
                    float v = transposed ? w[(((int64_t)ci * cout + co) * k + kh) * k + kw]
                                         : w[(((int64_t)co * cin + ci) * k + kh) * k + kw];
                    W0[(int64_t)co * per_co + (kh * k + kw) * cin_p + ci] = v;
                }

    if (form == 0) {
        double *out = (double *)malloc(sizeof(double) * cin_p);
        for (int co = 0; co < cout_p; ++co)
            for (int t = 0; t < taps; ++t) {
                const double *row = W0 + (int64_t)co * per_co + (int64_t)t * cin_p;
                block_transform_f64(H, hblock, row, out, 1, cin_p);
                for (int ci = 0; ci < cin_p; ++ci)
                    W1[(int64_t)co * per_co + (int64_t)t * cin_p + ci] = (float)out[ci];
            }
        free(out);
    } else {
        double *col = (double *)malloc(sizeof(double) * cout_p);
        double *out = (double *)malloc(sizeof(double) * cout_p);
        for (int64_t d = 0; d < per_co; ++d) {
            for (int co = 0; co < cout_p; ++co) col[co] = W0[(int64_t)co * per_co + d];
            block_transform_f64(H, hblock, col, out, 1, cout_p);
            for (int co = 0; co < cout_p; ++co) W1[(int64_t)co * per_co + d] = (float)out[co];
        }
        free(col);
        free(out);
    }

    if (w_real) memcpy(w_real, W1, sizeof(float) * (size_t)cout_p * per_co);
    for (int co = 0; co < cout_p; ++co) {
        const float *row = W1 + (int64_t)co * per_co;
        float A = 0.0f;
        for (int64_t d = 0; d < per_co; ++d)
            if (fabsf(row[d]) > A) A = fabsf(row[d]);
        const float s = A > 0.0f ? A / 127.0f : 1.0f;
        w_scale[co] = s;
        for (int64_t d = 0; d < per_co; ++d) {
            float t = nearbyintf(row[d] / s);
            if (t > 127.0f) t = 127.0f;
            if (t < -127.0f) t = -127.0f;
            wq[(int64_t)co * per_co + d] = (int8_t)t;
        }
    }

    if (form == 0) {
        for (int co = 0; co < cout_p; ++co) w_bias[co] = (bias && co < cout) ? bias[co] : 0.0f;
    } else {
        double *bb = (double *)calloc(cout_p, sizeof(double));
        double *out = (double *)malloc(sizeof(double) * cout_p);
        for (int co = 0; co < cout; ++co) bb[co] = bias ? bias[co] : 0.0;
        block_transform_f64(H, hblock, bb, out, 1, cout_p);
        for (int co = 0; co < cout_p; ++co) w_bias[co] = (float)out[co];
        free(bb);
        free(out);
    }
    free(W0);
    free(W1);
    free(H);
    return 0;
}

/* ------------------------------------------------------------------------- */
/* Output size of a convolution or transposed convolution.                    */
/* ------------------------------------------------------------------------- */
int orc_out_size(int in, int k, int stride, int pad, int transposed, int out_pad)
{
    if (transposed) return (in - 1) * stride - 2 * pad + k + out_pad;
    return (in + 2 * pad - k) / stride + 1;
}

/* Input row feeding output row o through tap i, or -1 when the tap lands on   */
/* zero padding.  Direct form: ih = o*s - p + i.  Transposed (gather) form:   */
/* t = o + p - i, used iff t >= 0, t % s == 0 and t/s < in.                   */
static int src_index(int o, int i, int in, int stride, int pad, int transposed)
{
    if (!transposed) {
        int ih = o * stride - pad + i;
        return (ih >= 0 && ih < in) ? ih : -1;
    }
    int t = o + pad - i;
    if (t < 0 || t % stride) return -1;
    t /= stride;
    return t < in ? t : -1;
}

/* ------------------------------------------------------------------------- */
/* O4. INT8 convolution with INT32 accumulation (Eq. integer_accumulation with */
/* zero points 0; Eq. linear_operator unfolded): a direct seven-loop sum.     */
/* xq: [n][h][w][cin_p] int8, wq: [cout_p][k][k][cin_p] int8 (OHWI),          */
/* acc: [n][ho][wo][cout_p] int32.  Out-of-range taps contribute 0.           */
/* ------------------------------------------------------------------------- */
/* zx: NULL, or one activation zero point per sample: the sum then runs over */
/* the centered codes x - z_x (Eq. integer_accumulation with z_w = 0), and    */
/* input pixels outside the image contribute nothing (the value zero).        */
void orc_conv_int8(const int8_t *xq, const int32_t *zx, int n, int h, int w, int cin_p,
                   const int8_t *wq, int cout_p, int k, int stride, int pad,
                   int transposed, int out_pad, int32_t *acc)
{
    const int ho = orc_out_size(h, k, stride, pad, transposed, out_pad);
    const int wo = orc_out_size(w, k, stride, pad, transposed, out_pad);
    #pragma omp parallel for collapse(2) schedule(dynamic)
    for (int b = 0; b < n; ++b)
        for (int oh = 0; oh < ho; ++oh)
            for (int ow = 0; ow < wo; ++ow)
                for (int co = 0; co < cout_p; ++co) {
                    const int32_t z = zx ? zx[b] : 0;
                    int32_t a = 0;
                    for (int kh = 0; kh < k; ++kh) {
                        const int ih = src_index(oh, kh, h, stride, pad, transposed);
                        if (ih < 0) continue;
                        for (int kw = 0; kw < k; ++kw) {
                            const int iw = src_index(ow, kw, w, stride, pad, transposed);
                            if (iw < 0) continue;
                            const int8_t *xp = xq + (((int64_t)b * h + ih) * w + iw) * cin_p;
                            const int8_t *wp = wq + (((int64_t)co * k + kh) * k + kw) * cin_p;
                            for (int ci = 0; ci < cin_p; ++ci)
                                a += ((int32_t)xp[ci] - z) * (int32_t)wp[ci];
                        }
                    }
                    acc[(((int64_t)b * ho + oh) * wo + ow) * cout_p + co] = a;
                }
}

/* Same loops in fp64 on real values: used for the unquantized function-       */
/* preservation checks.  x: [n][h][w][cin], wf: [cout][k][k][cin] (OHWI).     */
void orc_conv_f64(const double *x, int n, int h, int w, int cin,
                  const double *wf, int cout, int k, int stride, int pad,
                  int transposed, int out_pad, double *y)
{
    const int ho = orc_out_size(h, k, stride, pad, transposed, out_pad);
    const int wo = orc_out_size(w, k, stride, pad, transposed, out_pad);
    #pragma omp parallel for collapse(2) schedule(dynamic)
    for (int b = 0; b < n; ++b)
        for (int oh = 0; oh < ho; ++oh)
            for (int ow = 0; ow < wo; ++ow)
                for (int co = 0; co < cout; ++co) {
                    double a = 0.0;
                    for (int kh = 0; kh < k; ++kh) {
                        const int ih = src_index(oh, kh, h, stride, pad, transposed);
                        if (ih < 0) continue;
                        for (int kw = 0; kw < k; ++kw) {
                            const int iw = src_index(ow, kw, w, stride, pad, transposed);
                            if (iw < 0) continue;
                            const double *xp = x + (((int64_t)b * h + ih) * w + iw) * cin;
                            const double *wp = wf + (((int64_t)co * k + kh) * k + kw) * cin;
                            for (int ci = 0; ci < cin; ++ci) a += xp[ci] * wp[ci];
                        }
                    }
                    y[(((int64_t)b * ho + oh) * wo + ow) * cout + co] = a;
                }
}

/* ------------------------------------------------------------------------- */
/* O5. Epilogues.  acc: [n][pix][cout_p] int32, sx[n], sw[cout_p], bias.       */
/* DH: y = fma(float(acc), t_c, bias_c),  t_c = fl(fl(sx*sw_c) / b) (an exact */
/*     scaling when b is a power of two), for c < cout (output in the         */
/*     original basis, Eq. supp_padded_dh).                                   */
/* WH: z_c = fma(float(acc_c), fl(sx*sw_c), b~_c) for every c < cout_p (scale  */
/*     aligned before the basis change), then y = fl32(B_Cout^T z / b) with a */
/*     dense fp64 multiply, truncated to cout (Eq. supp_padded_wh).           */
/* ------------------------------------------------------------------------- */
int orc_epilogue(const int32_t *acc, int n, int64_t pix, int cout, int cout_p, int form,
                 int hblock, const float *sx, const float *sw, const float *bias, float *y)
{
    if (!supported(hblock) || (form == 1 && cout_p % hblock)) return -1;
    int8_t *H = NULL;
    if (form == 1) {
        /* the restore multiplies by the transpose (B^T B = b I; Sylvester   */
        /* blocks are symmetric, Paley-I blocks are not)                      */
        int8_t *Hf = (int8_t *)malloc((size_t)hblock * hblock);
        H = (int8_t *)malloc((size_t)hblock * hblock);
        orc_hadamard(hblock, Hf);
        for (int i = 0; i < hblock; ++i)
            for (int j = 0; j < hblock; ++j) H[i * hblock + j] = Hf[j * hblock + i];
        free(Hf);
    }
    for (int b = 0; b < n; ++b) {
        #pragma omp parallel
        {
            double *z = (double *)malloc(sizeof(double) * cout_p);
            double *out = (double *)malloc(sizeof(double) * cout_p);
            #pragma omp for schedule(static)
            for (int64_t p = 0; p < pix; ++p) {
                const int32_t *a = acc + ((int64_t)b * pix + p) * cout_p;
                float *yo = y + ((int64_t)b * pix + p) * cout;
                if (form == 0) {
                    for (int c = 0; c < cout; ++c) {
                        const float t = (sx[b] * sw[c]) / (float)hblock;   /* exact scaling for 2^k */
                        yo[c] = fmaf((float)a[c], t, bias[c]);
                    }
                } else {
                    for (int c = 0; c < cout_p; ++c)
                        z[c] = (double)fmaf((float)a[c], sx[b] * sw[c], bias[c]);
                    block_transform_f64(H, hblock, z, out, 1, cout_p);
                    for (int c = 0; c < cout; ++c) yo[c] = (float)(out[c] / (double)hblock);
                }
            }
            free(z);
            free(out);
        }
    }
    free(H);
    return 0;
}

/* The WH layer's dequantized accumulators before the output restore: O5's   */
/* z_c = fma(float(acc_c), fl(sx*sw_c), b~_c) for every c < cout_p.  When the */
/* next operand's transform uses the same blocks, B_next y = B B^T z / b = z  */
/* on every kept block in exact arithmetic (Table I: the WH output transform  */
/* and the next DH input transform cancel), so z is that next operand.        */
void orc_wh_z(const int32_t *acc, int n, int64_t pix, int cout_p, const float *sx, const float *sw,
              const float *bias, float *z)
{
    for (int b = 0; b < n; ++b)
        for (int64_t p = 0; p < pix; ++p)
            for (int c = 0; c < cout_p; ++c) {
                const int64_t i = ((int64_t)b * pix + p) * cout_p + c;
                z[i] = fmaf((float)acc[i], sx[b] * sw[c], bias[c]);
            }
}

/* ------------------------------------------------------------------------- */
/* O6. Integer-only inter-layer transition (Eq. integer_accumulation with    */
/* zero points 0, Eq. integer_fixed_point_scale, Eq. integer_hadamard_        */
/* transition, Table I), static scales.  In the unnormalized transforms used */
/* throughout, one accumulator step of channel c is worth                     */
/*   u_c = s_x s_w,c / beta_in    (beta_in = block of a DH layer's input       */
/*                                 transform, 1 for WH),                      */
/* and the output transform of a WH layer divides by its block beta_out      */
/* (1 for DH), so the bias in accumulator steps and the scale ratio are       */
/*   b_int,c = rne(b_c / u_c),  rho_c = u_c / (beta_out s_y),                 */
/*   M_c = rne(2^n rho_c),                                                    */
/* with the shared shift n the largest in [0, 62] that keeps every M_c at or  */
/* below M_max = floor(2^62 / (A_max G)), A_max = K 127^2 + max|b_int| the    */
/* accumulator bound and G the product of the transform gains (block size of  */
/* the WH output transform, block size of the next DH input transform).       */
/* Returns n, or -1 when no n >= 0 fits (or |b_int| >= 2^30).                 */
/* ------------------------------------------------------------------------- */
int orc_int_requant_params(int cout_p, float s_x, const float *s_w, const float *bias, float s_y,
                           int beta_in, int beta_out, int K, int gain, int32_t *M, int32_t *b_int)
{
    if (beta_in < 1 || beta_out < 1 || gain < 1) return -1;
    double bmax = 0.0;
    for (int c = 0; c < cout_p; ++c) {
        const double u = (double)s_x * (double)s_w[c] / (double)beta_in;   /* exact: product, power of two */
        const double bi = rint((double)bias[c] / u);
        if (fabs(bi) >= 1073741824.0) return -1;
        b_int[c] = (int32_t)bi;
        if (fabs(bi) > bmax) bmax = fabs(bi);
    }
    const double amax = (double)K * 127.0 * 127.0 + bmax;
    double mmax = floor(4611686018427387904.0 / (amax * (double)gain));   /* 2^62 / (A_max G) */
    if (mmax > 2147483647.0) mmax = 2147483647.0;
    for (int n = 62; n >= 0; --n) {
        int ok = 1;
        for (int c = 0; c < cout_p && ok; ++c) {
            const double rho = (double)s_x * (double)s_w[c] / ((double)beta_in * (double)beta_out * (double)s_y);
            if (rint(ldexp(rho, n)) > mmax) ok = 0;
        }
        if (!ok) continue;
        for (int c = 0; c < cout_p; ++c) {
            const double rho = (double)s_x * (double)s_w[c] / ((double)beta_in * (double)beta_out * (double)s_y);
            M[c] = (int32_t)rint(ldexp(rho, n));
        }
        return n;
    }
    return -1;
}

/* rne(w / 2^n) for an integer w: the exact quotient rounded half to even. */
static int64_t rne_shift(int64_t w, int n)
{
    if (n == 0) return w;
    const int64_t p = (int64_t)1 << n;
    int64_t q = w / p;                                /* truncated toward zero */
    if (w % p != 0 && w < 0) q -= 1;                  /* floor */
    const int64_t r = w - q * p;                      /* 0 <= r < 2^n */
    const int64_t half = (int64_t)1 << (n - 1);
    if (r > half || (r == half && (q & 1))) return q + 1;
    return q;
}

/* The transition itself on accumulators acc [P][cout_p]:                     */
/*   a'  = acc + b_int;  v = H_out(M (.) a') (WH: blocks of wb over cout_p;    */
/*   wb = 1: identity), truncated to cout;  w = H_in(v) (DH next: blocks of    */
/*   nb over cout, cout % nb == 0; nb = 1: identity);                         */
/*   q = clamp(rne(w / 2^n), -127, 127).  All in int64 with dense matrices.    */
int orc_int_transition(const int32_t *acc, int64_t P, int cout, int cout_p, const int32_t *M,
                       const int32_t *b_int, int n, int wb, int nb, int8_t *q)
{
    if (!supported(wb) || !supported(nb) || cout_p % wb || cout % nb || n < 0 || n > 62) return -1;
    int8_t *Ho = (int8_t *)malloc((size_t)wb * wb);
    int8_t *Hi = (int8_t *)malloc((size_t)nb * nb);
    orc_hadamard(wb, Ho);               /* Sylvester for powers of two */
    orc_hadamard(nb, Hi);
    #pragma omp parallel
    {
        int64_t *p = (int64_t *)malloc(sizeof(int64_t) * cout_p);
        int64_t *v = (int64_t *)malloc(sizeof(int64_t) * cout_p);
        #pragma omp for schedule(static)
        for (int64_t px = 0; px < P; ++px) {
            const int32_t *a = acc + px * cout_p;
            for (int c = 0; c < cout_p; ++c) p[c] = (int64_t)M[c] * ((int64_t)a[c] + b_int[c]);
            /* the WH output restore multiplies by the transposed block (B^T B = b I) */
            for (int blk = 0; blk < cout_p; blk += wb)
                for (int i = 0; i < wb; ++i) {
                    int64_t s = 0;
                    for (int j = 0; j < wb; ++j) s += Ho[j * wb + i] * p[blk + j];
                    v[blk + i] = s;
                }
            for (int blk = 0; blk < cout; blk += nb)
                for (int i = 0; i < nb; ++i) {
                    int64_t s = 0;
                    for (int j = 0; j < nb; ++j) s += Hi[i * nb + j] * v[blk + j];
                    int64_t r = rne_shift(s, n);
                    if (r > 127) r = 127;
                    if (r < -127) r = -127;
                    q[px * cout + blk + i] = (int8_t)r;
                }
        }
        free(p);
        free(v);
    }
    free(Ho);
    free(Hi);
    return 0;
}

/* ------------------------------------------------------------------------- */
/* O7. Range-expansion profiling (Eq. hadamard_sensitivity) and the form     */
/* rule (Eq. layerwise_hadamard_selection).                                   */
/* For sample k of x [n][P][C] (its pixels padded with zero channels to a     */
/* multiple of b): ax[k] = max |x|, ah[k] = max |S| with S = fl32(B_C x_pad)  */
/* as in O3 (the unnormalized transform the activation quantizer sees).  The */
/* paper compares the orthonormal transform H = B / sqrt(b) against x, so    */
/* the sample expands iff ah > sqrt(b) ax, decided exactly as                 */
/*   ah^2 > b ax^2   in fp64 (squares of fp32 values and their products by a  */
/*                    power of two are exact in fp64).                        */
/* ------------------------------------------------------------------------- */
int orc_range_expansion(const float *x, int n, int64_t P, int C, int b, float *ax, float *ah, int32_t *flags)
{
    if (!supported(b) || C <= 0 || n <= 0 || P <= 0) return -1;
    const int Cp = round_up(C, b);
    int8_t *H = (int8_t *)malloc((size_t)b * b);
    orc_hadamard(b, H);                 /* Sylvester for a power of two */
    for (int k = 0; k < n; ++k) {
        const float *xs = x + (int64_t)k * P * C;
        float mx = 0.0f, mh = 0.0f;
        #pragma omp parallel reduction(max : mx, mh)
        {
            double *in = (double *)malloc(sizeof(double) * Cp);
            double *out = (double *)malloc(sizeof(double) * Cp);
            #pragma omp for schedule(static)
            for (int64_t p = 0; p < P; ++p) {
                for (int c = 0; c < Cp; ++c) {
                    in[c] = c < C ? (double)xs[p * C + c] : 0.0;
                    if (c < C && fabsf(xs[p * C + c]) > mx) mx = fabsf(xs[p * C + c]);
                }
                block_transform_f64(H, b, in, out, 1, Cp);
                for (int c = 0; c < Cp; ++c) {
                    const float v = fabsf((float)out[c]);
                    if (v > mh) mh = v;
                }
            }
            free(in);
            free(out);
        }
        ax[k] = mx;
        ah[k] = mh;
        flags[k] = (double)mh * (double)mh > (double)b * ((double)mx * (double)mx);
    }
    free(H);
    return 0;
}

/* pi = WH (1) if p = expansions / images > tau, else DH (0); p is the       */
/* correctly rounded fp64 quotient.  -1 for images <= 0 or a count outside    */
/* [0, images].                                                               */
int orc_select_form(int64_t expansions, int64_t images, double tau)
{
    if (images <= 0 || expansions < 0 || expansions > images) return -1;
    const double p = (double)expansions / (double)images;
    return p > tau ? 1 : 0;
}
