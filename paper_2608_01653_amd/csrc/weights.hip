// Offline weight preparation on the device (step a1).
//
// DH (Eq. hadamard_linear_equivalence, Eq. supp_padded_dh): every (co, tap) row
// of the contraction is multiplied by B_Cin = I (x) H~_b (H~_b Sylvester, or the
// Kronecker order P (x) H~_16 for b = 192, 320; then W' = W B^T).  WH (Eq.
// weight_only_hadamard_equivalence, Eq. supp_padded_wh_parameters): every (tap, ci)
// column is multiplied by B_Cout, and the bias becomes b~ = B_Cout [b; 0].
// Each transformed value is an fp64 sum over j = 0..b-1 in ascending order of
// (-1)^popcount(i & j) * w_j (products with +-1 are exact), rounded once to fp32.
// Then per output channel s_w = fl32(max|W'| / 127) (1 if the row is zero) and
// q = clamp(rne(fl32(W' / s_w)), -127, 127) with IEEE fp32 division
// (Eq. symmetric_q, per-output-channel weights).
#include "hatq_device.h"
#include "hatq_launch.h"

namespace hatq {
namespace {

constexpr int kThreads = 256;

// Original weight W0[co][kh][kw][ci] read from the PyTorch layout, 0 outside.
__device__ __forceinline__ double w_orig(const PrepArgs &a, int co, int tap, int ci) {
    if (co >= a.cout || ci >= a.cin) return 0.0;
    const int kh = tap / a.k, kw = tap - kh * a.k;
    const int64_t idx = a.transposed ? (((int64_t)ci * a.cout + co) * a.k + kh) * a.k + kw
                                     : (((int64_t)co * a.cin + ci) * a.k + kh) * a.k + kw;
    return (double)a.w[idx];
}

__device__ __forceinline__ double hsign(int i, int j) { return (__popc(i & j) & 1) ? -1.0 : 1.0; }

// Entry (i, j) of the order-b block: Sylvester for powers of two, else the
// Kronecker order P (x) H~_16 (index a*16 + l).
__device__ __forceinline__ double block_sign(int b, int i, int j) {
    const int q = kron_q(b);
    if (q == 0) return hsign(i, j);
    return paley1_entry(q, i >> 4, j >> 4) * hsign(i & 15, j & 15);
}

// Transformed weight W'[co][d], d = tap*cin_p + ci.
__device__ float w_prime(const PrepArgs &a, int co, int d) {
    const int tap = d / a.cin_p, ci = d - tap * a.cin_p;
    const int b = a.hblock;
    double acc = 0.0;
    if (a.form == 0) {
        const int blk = ci / b * b, i = ci - blk;
        for (int j = 0; j < b; ++j) acc += block_sign(b, i, j) * w_orig(a, co, tap, blk + j);
    } else {
        const int blk = co / b * b, i = co - blk;
        for (int j = 0; j < b; ++j) acc += block_sign(b, i, j) * w_orig(a, blk + j, tap, ci);
    }
    return (float)acc;
}

// K-blocked copy of one channel's codes: contraction byte d' goes to
// wpack[d'/64][co][d'%64].  Natural order d' = d, except for row-run layers,
// whose kernel contracts one 16-byte run per kernel row: d' = 16*kh + j holds
// d = kh*k*cin_p + j for j < k*cin_p and 0 otherwise.
__device__ void pack_row(const PrepArgs &a, int co, const int8_t *row) {
    for (int dp = threadIdx.x; dp < a.pack_stride; dp += kThreads) {
        int d = dp;
        if (a.rowrun) {
            const int kh = dp >> 4, j = dp & 15;
            d = (kh < a.k && j < a.k * a.cin_p) ? kh * a.k * a.cin_p + j : a.k_stride;
        }
        a.wpack[((int64_t)(dp >> 6) * a.cout_p + co) * 64 + (dp & 63)] = d < a.k_stride ? row[d] : (int8_t)0;
    }
}

__global__ void __launch_bounds__(kThreads) pack_kernel(const PrepArgs a) {
    pack_row(a, blockIdx.x, a.wq + (int64_t)blockIdx.x * a.k_stride);
}

__global__ void __launch_bounds__(kThreads) prepare_kernel(const PrepArgs a) {
    const int co = blockIdx.x;
    float m = 0.0f;
    for (int d = threadIdx.x; d < a.k_total; d += kThreads) m = fmaxf(m, fabsf(w_prime(a, co, d)));
    m = wave_max(m);
    __shared__ float red[kThreads / 64];
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
    __syncthreads();
    float A = red[0];
#pragma unroll
    for (int k = 1; k < kThreads / 64; ++k) A = fmaxf(A, red[k]);
    const float s = A > 0.0f ? A / 127.0f : 1.0f;
    int8_t *row = a.wq + (int64_t)co * a.k_stride;
    for (int d = threadIdx.x; d < a.k_stride; d += kThreads) {
        int8_t q = 0;
        if (d < a.k_total) q = (int8_t)(int)rintf(clamp127(w_prime(a, co, d) / s));
        row[d] = q;
    }
    __syncthreads();   // this block's wq row is complete
    pack_row(a, co, row);
    if (threadIdx.x == 0) {
        a.w_scale[co] = s;
        double bv = 0.0;
        if (a.bias) {
            if (a.form == 0) {
                bv = co < a.cout ? (double)a.bias[co] : 0.0;
            } else {
                const int b = a.hblock, blk = co / b * b, i = co - blk;
                for (int j = 0; j < b; ++j)
                    bv += block_sign(b, i, j) * (blk + j < a.cout ? (double)a.bias[blk + j] : 0.0);
            }
        }
        a.w_bias[co] = (float)bv;
    }
}

// Integer transition parameters (Eq. integer_accumulation, Eq.
// integer_fixed_point_scale), one block.  One accumulator step of channel c is
// u_c = s_x s_w,c / beta_in (exact: a product of two floats over a power of
// two), so b_int,c = rne(b_c / u_c); the scale ratio rho_c = u_c / (beta_out
// s_y) becomes M_c = rne(2^n rho_c) with the shared shift n, the largest in
// [0, 62] that keeps every M_c at or below floor(2^62 / (A_max G)) (and below
// 2^31), A_max = K 127^2 + max |b_int| bounding |acc + b_int| and G the gain of
// the two transforms, so every int64 partial sum of the transition is exact.
// fp64 with correctly rounded division throughout; |b_int| >= 2^30 or no
// fitting n gives n = -1.
__global__ void __launch_bounds__(kThreads) int_params_kernel(const IntParamArgs a) {
    __shared__ double s_bmax[kThreads];
    __shared__ int s_n[kThreads];
    const int tid = threadIdx.x;
    double bmax = 0.0;
    for (int c = tid; c < a.cout_p; c += kThreads) {
        const double u = (double)a.s_x * (double)a.w_scale[c] / (double)a.beta_in;
        const double bi = rint((double)a.bias[c] / u);
        const bool big = !(fabs(bi) < 1073741824.0);   // also catches NaN
        a.table[a.cout_p + c] = big ? 0 : (int32_t)bi;
        bmax = fmax(bmax, big ? INFINITY : fabs(bi));
    }
    s_bmax[tid] = bmax;
    __syncthreads();
    for (int h = kThreads / 2; h > 0; h >>= 1) {
        if (tid < h) s_bmax[tid] = fmax(s_bmax[tid], s_bmax[tid + h]);
        __syncthreads();
    }
    const double bm = s_bmax[0];
    const double amax = (double)a.K * 127.0 * 127.0 + bm;
    double mmax = floor(4611686018427387904.0 / (amax * (double)a.gain));
    if (mmax > 2147483647.0) mmax = 2147483647.0;
    const double den = (double)a.beta_in * (double)a.beta_out * (double)a.s_y;
    int nmin = bm < 1073741824.0 ? 62 : -1;
    for (int c = tid; c < a.cout_p; c += kThreads) {
        const double rho = (double)a.s_x * (double)a.w_scale[c] / den;
        int n = nmin;
        while (n >= 0 && rint(ldexp(rho, n)) > mmax) --n;
        nmin = n;
    }
    s_n[tid] = nmin;
    __syncthreads();
    for (int h = kThreads / 2; h > 0; h >>= 1) {
        if (tid < h) s_n[tid] = min(s_n[tid], s_n[tid + h]);
        __syncthreads();
    }
    const int n = s_n[0];
    for (int c = tid; c < a.cout_p; c += kThreads) {
        const double rho = (double)a.s_x * (double)a.w_scale[c] / den;
        a.table[c] = n >= 0 ? (int32_t)rint(ldexp(rho, n)) : 0;
    }
    if (tid == 0) a.table[2 * a.cout_p] = n;
}

// One block per output channel, one thread per tap (k*k <= kMaxTaps <= the
// block), then the block's total.
__global__ void __launch_bounds__(kThreads) tapsum_kernel(const PrepArgs a, int32_t *tapsum) {
    __shared__ int32_t s_sum[kThreads];
    const int c = blockIdx.x, t = threadIdx.x;
    const int taps = a.k * a.k;
    int32_t sum = 0;
    if (t < taps) {
        const int8_t *row = a.wq + (int64_t)c * a.k_stride + t * a.cin_p;
        for (int ci = 0; ci < a.cin_p; ++ci) sum += row[ci];
        tapsum[(int64_t)t * a.cout_p + c] = sum;
    }
    s_sum[t] = sum;
    __syncthreads();
    for (int h = kThreads / 2; h > 0; h >>= 1) {
        if (t < h) s_sum[t] += s_sum[t + h];
        __syncthreads();
    }
    if (t == 0) tapsum[(int64_t)taps * a.cout_p + c] = s_sum[0];
}

}  // namespace

hipError_t launch_tapsums(const PrepArgs &a, int32_t *tapsum, hipStream_t st) {
    if (a.k * a.k > kThreads) return hipErrorInvalidValue;
    tapsum_kernel<<<a.cout_p, kThreads, 0, st>>>(a, tapsum);
    return hipGetLastError();
}

hipError_t launch_int_params(const IntParamArgs &a, hipStream_t st) {
    int_params_kernel<<<1, kThreads, 0, st>>>(a);
    return hipGetLastError();
}

hipError_t launch_prepare(const PrepArgs &a, hipStream_t st) {
    prepare_kernel<<<a.cout_p, kThreads, 0, st>>>(a);
    return hipGetLastError();
}

hipError_t launch_pack(const PrepArgs &a, hipStream_t st) {
    pack_kernel<<<a.cout_p, kThreads, 0, st>>>(a);
    return hipGetLastError();
}

}  // namespace hatq
