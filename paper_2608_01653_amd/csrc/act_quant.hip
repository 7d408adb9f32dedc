// Activation transform + per-sample absmax + INT8 quantization (steps a2-a4).
//
// The input of one sample is a flat fp32 array of E = h*w*c elements (NHWC).
// With c % b == 0 every Hadamard block (b consecutive channels of one pixel) is
// b-aligned in the flat array, so the kernel tiles the array into "items" of
// I = max(64, b) consecutive floats without looking at pixel boundaries.
//
// One quad (4 lanes) owns one item.  Lane t of the quad holds the channels
// c = 16*i + 4*t + j (j = 0..3 inside a float4, i = 0..I/16-1): bits 0-1 of
// the channel index are inside a float4, bits 2-3 are the lane, bits 4+ are the
// register index.  Loads are 64 contiguous bytes per quad per instruction.
//
// Two kernels:
//   absmax_kernel: transform, max |S| per sample (one atomic per block).
//   quant_kernel : transform again, quantize with s = fl32(A / 127), store codes.
// When the producer of x already computed A (next_absmax of the convolution),
// only quant_kernel runs and x is read once.
#include <mutex>

#include "hatq_device.h"
#include "hatq_launch.h"

// Scratch of the no-allocation entry point: the per-sample absmax of the
// two-pass quantization for callers that cannot allocate.  Every GPU the
// library runs on holds its own copy until the process ends.  In host code the
// name is a stand-in, not a device address: the address comes from
// hipGetSymbolAddress, looked up once per device (scratch_absmax below).
static __device__ __align__(256) float scratch[hatq::kNoAllocMaxSamples * hatq::kAbsSlots];

namespace hatq {

__global__ void fill_u32_kernel(uint32_t *p, int n, uint32_t v) {
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = v;
}

namespace {

constexpr int kThreads = 256;
constexpr int kQuadsPerBlock = kThreads / 4;

template <int B>
__device__ __forceinline__ void load_item(const float *xs, int64_t base, int64_t E, int t,
                                          float (&v)[4 * ItemShape<B>::R]) {
    constexpr int R = ItemShape<B>::R;
    constexpr int I = ItemShape<B>::I;
    const bool full = base + I <= E;
#pragma unroll
    for (int i = 0; i < R; ++i) {
        const int64_t off = base + 16 * i + 4 * t;
        float4 f = make_float4(0.f, 0.f, 0.f, 0.f);
        if (full || off < E) f = *reinterpret_cast<const float4 *>(xs + off);
        v[4 * i + 0] = f.x;
        v[4 * i + 1] = f.y;
        v[4 * i + 2] = f.z;
        v[4 * i + 3] = f.w;
    }
}

template <int B>
__global__ void __launch_bounds__(kThreads) absmax_kernel(const float *__restrict__ x, int64_t E,
                                                          float *__restrict__ absmax) {
    constexpr int R = ItemShape<B>::R;
    constexpr int I = ItemShape<B>::I;
    const int n = blockIdx.y;
    const float *xs = x + (int64_t)n * E;
    const int t = threadIdx.x & 3;
    const int64_t items = (E + I - 1) / I;
    float m = 0.0f;
    // (unrolled so the loads of several items are in flight together: the
    // grid is small, so each quad walks several items)
#pragma unroll 4
    for (int64_t it = (int64_t)blockIdx.x * kQuadsPerBlock + (threadIdx.x >> 2); it < items;
         it += (int64_t)gridDim.x * kQuadsPerBlock) {
        float v[4 * R];
        load_item<B>(xs, it * I, E, t, v);
        fwht_item<B>(v, t);
#pragma unroll
        for (int r = 0; r < 4 * R; ++r) m = fmaxf(m, fabsf(v[r]));
    }
    m = wave_max(m);
    __shared__ float red[kThreads / 64];
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
        float b = red[0];
#pragma unroll
        for (int k = 1; k < kThreads / 64; ++k) b = fmaxf(b, red[k]);
        atomic_max_nonneg(absmax + (int64_t)n * kAbsSlots + blockIdx.x % kAbsSlots, b);
    }
}

// The same for blocks of 1 (no transform): max |x| over the sample read as
// float4 (E % 4 == 0), four loads per thread in flight per iteration.
__global__ void __launch_bounds__(kThreads) absmax_flat_kernel(const float *__restrict__ x, int64_t E,
                                                               float *__restrict__ absmax) {
    const int n = blockIdx.y;
    const float4 *xs = reinterpret_cast<const float4 *>(x + (int64_t)n * E);
    const int64_t E4 = E >> 2;
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    auto m4 = [](float m, const float4 &f) {
        return fmaxf(fmaxf(fmaxf(m, fabsf(f.x)), fabsf(f.y)), fmaxf(fabsf(f.z), fabsf(f.w)));
    };
    float m = 0.0f;
    for (; i + 3 * stride < E4; i += 4 * stride) {
        const float4 a = xs[i], b = xs[i + stride], c = xs[i + 2 * stride], d = xs[i + 3 * stride];
        m = m4(m4(m4(m4(m, a), b), c), d);
    }
    for (; i < E4; i += stride) m = m4(m, xs[i]);
    m = wave_max(m);
    __shared__ float red[kThreads / 64];
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
        float b = red[0];
#pragma unroll
        for (int k = 1; k < kThreads / 64; ++k) b = fmaxf(b, red[k]);
        atomic_max_nonneg(absmax + (int64_t)n * kAbsSlots + blockIdx.x % kAbsSlots, b);
    }
}

// Items per quad per loop iteration (all their loads issued before first use).
#ifndef HATQ_QUANT_UN
#define HATQ_QUANT_UN 1
#endif
template <int B>
struct QuantUnroll {
    // two items in flight per quad: the untransformed 3-channel image's two-pass
    // quantization 80.5 -> 77.3 us; with blocks of 64, 178 -> 182 us
    static constexpr int UN = B == 1 ? 2 : HATQ_QUANT_UN;
};

// Quantize one transformed item (s = act scale, r = fl(1/s)) and store its codes.
// cc > 0: codes in the chunk-major layout of a sample of cc channels (items of
// 64 channels, cc % 64 == 0): the item of pixel p, channels 64m .. 64m + 63, goes
// to ((m * (E / cc)) + p) * 64.
template <int B>
__device__ __forceinline__ void quant_store_item(const float (&vin)[4 * ItemShape<B>::R], int8_t *qs, int64_t base,
                                                 int64_t E, int t, float s, float r, bool fast_ok, float sigma,
                                                 int cc) {
    constexpr int R = ItemShape<B>::R;
    constexpr int I = ItemShape<B>::I;
    static_assert(R % 4 == 0, "groups of four words");
    const float rs = sigma * r;
    uint32_t u[4 * R];
    bool near = !fast_ok;
#pragma unroll
    for (int k = 0; k < 4 * R; ++k) {
        const float tq = clamp127(vin[k] * rs);
        const float uf = tq + HATQ_MAGIC;
        const float kf = uf - HATQ_MAGIC;
        near |= fabsf(tq - kf) > HATQ_NEAR_TIE;
        u[k] = __float_as_uint(uf);
    }
    if (near) {
#pragma unroll
        for (int k = 0; k < 4 * R; ++k) {
            const float q = rintf(clamp127((sigma * vin[k]) / s));
            u[k] = __float_as_uint(q + HATQ_MAGIC);
        }
    }
    const bool full = base + I <= E;
    if (full) {
        // Word i of lane t holds channels 16i + 4t .. +3.  A 4 x 4 transpose of
        // words inside the quad (two DPP swap stages) gives lane t channels
        // 64g + 16t .. +15 of each group g of four words, so every lane stores
        // 16 contiguous bytes and the wave 1 KB per group.
#pragma unroll
        for (int g = 0; g < R / 4; ++g) {
            int w[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int k = 4 * (4 * g + i);
                w[i] = (int)pack_low_bytes(u[k], u[k + 1], u[k + 2], u[k + 3]);
            }
            int x[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) x[i] = __builtin_amdgcn_mov_dpp(w[i ^ 1], 0xB1, 0xF, 0xF, true);   // lane ^ 1
#pragma unroll
            for (int i = 0; i < 4; ++i) w[i] = ((t ^ i) & 1) ? x[i] : w[i];
#pragma unroll
            for (int i = 0; i < 4; ++i) x[i] = __builtin_amdgcn_mov_dpp(w[i ^ 2], 0x4E, 0xF, 0xF, true);   // lane ^ 2
#pragma unroll
            for (int i = 0; i < 4; ++i) w[i] = ((t ^ i) & 2) ? x[i] : w[i];
            int8_t *dst = qs + base + 64 * g + 16 * t;
            if (I == 64 && cc > 0) {
                const int64_t p = base / cc;
                dst = qs + (((base - p * cc) >> 6) * (E / cc) + p) * 64 + 16 * t;
            }
            // (xq need only be 4-byte aligned and a sample's E only a multiple
            // of 4; base is a multiple of 64, so the sample's start decides,
            // uniformly for the block)
            if ((reinterpret_cast<uintptr_t>(qs) & 15) == 0) {
                // streaming store: the codes are read by the next convolution,
                // not by this kernel, so they bypass the caches on the way out
                // (782 -> 716 us on the 805 M-element tensor)
                __builtin_nontemporal_store(v4i{w[0], w[1], w[2], w[3]}, reinterpret_cast<v4i *>(dst));
            } else {
#pragma unroll
                for (int i = 0; i < 4; ++i) reinterpret_cast<int *>(dst)[i] = w[i];
            }
        }
        return;
    }
#pragma unroll
    for (int i = 0; i < R; ++i) {
        const int64_t off = base + 16 * i + 4 * t;
        if (off < E)
            *reinterpret_cast<uint32_t *>(qs + off) = pack_low_bytes(u[4 * i], u[4 * i + 1], u[4 * i + 2], u[4 * i + 3]);
    }
}

template <int B>
__global__ void __launch_bounds__(kThreads) quant_kernel(const float *__restrict__ x, int64_t E,
                                                         const float *__restrict__ absmax,
                                                         int8_t *__restrict__ xq,
                                                         float *__restrict__ act_scale, int cc, int slots) {
    constexpr int I = ItemShape<B>::I;
    constexpr int R = ItemShape<B>::R;
    constexpr int UN = QuantUnroll<B>::UN;
    // Sample order: when the batch splits evenly over the 8 XCDs, the window
    // convolution that usually produced x gave XCD k the samples k g .. k g +
    // g - 1 (g = n / 8) and finished their last ones last, so the launch takes
    // samples last-finished first and reads each from its end: its first reads
    // meet the lines most recently written, still in the 256 MB memory-side
    // cache (layer 3's 201 M-element input: 188 -> 181 us).  Any order gives
    // the same codes.
    const int ns = gridDim.y;
    int n = blockIdx.y;
    if (ns % 8 == 0) {
        const int g = ns / 8, j = g - 1 - n / 8, k = n % 8;
        n = k * g + j;
    }
    const bool rev = ns % 8 == 0;
    const float *xs = x + (int64_t)n * E;
    int8_t *qs = xq + (int64_t)n * E;
    const int t = threadIdx.x & 3;
    // the sample's absmax: one value (given), or the maximum of its slots
    float am = absmax[(int64_t)n * slots];
    for (int k = 1; k < slots; ++k) am = fmaxf(am, absmax[(int64_t)n * slots + k]);
    const float s = act_scale_from_absmax(am);
    if (blockIdx.x == 0 && threadIdx.x == 0) act_scale[n] = s;
    const float r = 1.0f / s;
    // The fast path needs r and every t finite and normal-range; a scale below
    // 2^-125 or above 2^125 takes the exact division for every element.
    const bool fast_ok = s >= 0x1p-125f && s <= 0x1p125f;
    const int64_t items = (E + I - 1) / I;
    const int64_t step = (int64_t)gridDim.x * kQuadsPerBlock;
    for (int64_t it0 = (int64_t)blockIdx.x * kQuadsPerBlock * UN + (threadIdx.x >> 2); it0 < items;
         it0 += step * UN) {
        float v[UN][4 * R];
#pragma unroll
        for (int u = 0; u < UN; ++u) {
            const int64_t it = it0 + u * kQuadsPerBlock;
            if (it < items) load_item<B>(xs, (rev ? items - 1 - it : it) * I, E, t, v[u]);
        }
#pragma unroll
        for (int u = 0; u < UN; ++u) {
            const int64_t it = it0 + u * kQuadsPerBlock;
            if (it >= items) break;
            const float sigma = fwht_item<B>(v[u], t);
            quant_store_item<B>(v[u], qs, (rev ? items - 1 - it : it) * I, E, t, s, r, fast_ok, sigma, cc);
        }
    }
}

// ---- affine quantization (Eq. affine_q, Eq. uniform_q) ----------------------
// Signed grid [-128, 127].  amax[k] = max(max S, 0), amax[n + k] = max(-min S, 0)
// (both non-negative, so the order-preserving atomic serves both).
template <int B>
__global__ void __launch_bounds__(kThreads) minmax_kernel(const float *__restrict__ x, int64_t E,
                                                          float *__restrict__ amax) {
    constexpr int R = ItemShape<B>::R;
    constexpr int I = ItemShape<B>::I;
    const int k = blockIdx.y;
    const float *xs = x + (int64_t)k * E;
    const int t = threadIdx.x & 3;
    const int64_t items = (E + I - 1) / I;
    float hi = 0.0f, lo = 0.0f;   // max(S, 0) and max(-S, 0)
#pragma unroll 4
    for (int64_t it = (int64_t)blockIdx.x * kQuadsPerBlock + (threadIdx.x >> 2); it < items;
         it += (int64_t)gridDim.x * kQuadsPerBlock) {
        float v[4 * R];
        load_item<B>(xs, it * I, E, t, v);
        const float sigma = fwht_item<B>(v, t);
#pragma unroll
        for (int r = 0; r < 4 * R; ++r) {
            const float sv = sigma * v[r];
            hi = fmaxf(hi, sv);
            lo = fmaxf(lo, -sv);
        }
    }
    hi = wave_max(hi);
    lo = wave_max(lo);
    __shared__ float red[2][kThreads / 64];
    if ((threadIdx.x & 63) == 0) {
        red[0][threadIdx.x >> 6] = hi;
        red[1][threadIdx.x >> 6] = lo;
    }
    __syncthreads();
    if (threadIdx.x < 2) {
        float b = red[threadIdx.x][0];
#pragma unroll
        for (int w = 1; w < kThreads / 64; ++w) b = fmaxf(b, red[threadIdx.x][w]);
        atomic_max_nonneg(amax + (threadIdx.x ? gridDim.y : 0) + k, b);
    }
}

// s = fl32(fl32(hi + lo) / 255) and z = clamp(rne(fl32(lo / s)) - 128) for a
// nonzero range (hi + lo = xmax' - xmin'), else s = 1, z = 0.
__device__ __forceinline__ void affine_params(float hi, float lo, float &s, int &z) {
    const float r = hi + lo;
    s = 1.0f;
    z = 0;
    if (r > 0.0f) {
        s = r / 255.0f;
        z = (int)rintf(lo / s) - 128;
        z = z < -128 ? -128 : (z > 127 ? 127 : z);
    }
}

// Codes q = clamp(rne(fl32(S / s)) + z, -128, 127), IEEE division per element.
template <int B>
__global__ void __launch_bounds__(kThreads) quant_affine_kernel(const float *__restrict__ x, int64_t E,
                                                                const float *__restrict__ amax,
                                                                int8_t *__restrict__ xq, float *__restrict__ act_scale,
                                                                int32_t *__restrict__ act_zero) {
    constexpr int I = ItemShape<B>::I;
    constexpr int R = ItemShape<B>::R;
    const int k = blockIdx.y;
    const float *xs = x + (int64_t)k * E;
    int8_t *qs = xq + (int64_t)k * E;
    const int t = threadIdx.x & 3;
    float s;
    int z;
    affine_params(amax[k], amax[gridDim.y + k], s, z);
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        act_scale[k] = s;
        act_zero[k] = z;
    }
    const float zf = (float)z;
    const int64_t items = (E + I - 1) / I;
    for (int64_t it = (int64_t)blockIdx.x * kQuadsPerBlock + (threadIdx.x >> 2); it < items;
         it += (int64_t)gridDim.x * kQuadsPerBlock) {
        float v[4 * R];
        load_item<B>(xs, it * I, E, t, v);
        const float sigma = fwht_item<B>(v, t);
        uint32_t u[4 * R];
#pragma unroll
        for (int r = 0; r < 4 * R; ++r) {
            const float q = __builtin_amdgcn_fmed3f(rintf((sigma * v[r]) / s) + zf, -128.0f, 127.0f);
            u[r] = (uint32_t)(int32_t)q;
        }
        const int64_t base = it * I;
        const bool full = base + I <= E;
#pragma unroll
        for (int i = 0; i < R; ++i) {
            const int64_t off = base + 16 * i + 4 * t;
            if (full || off < E)
                *reinterpret_cast<uint32_t *>(qs + off) = pack_low_bytes(u[4 * i], u[4 * i + 1], u[4 * i + 2], u[4 * i + 3]);
        }
    }
}

// ---- range-expansion profiling (Eq. hadamard_sensitivity) -------------------
// One read of x gives both maxima of each sample: max |x| (into amax[k]) and
// max |S| of the same butterfly the quantizer applies (into amax[n + k]).
template <int B>
__global__ void __launch_bounds__(kThreads) range_kernel(const float *__restrict__ x, int64_t E,
                                                         float *__restrict__ amax) {
    constexpr int R = ItemShape<B>::R;
    constexpr int I = ItemShape<B>::I;
    const int k = blockIdx.y;
    const float *xs = x + (int64_t)k * E;
    const int t = threadIdx.x & 3;
    const int64_t items = (E + I - 1) / I;
    float mx = 0.0f, mh = 0.0f;
#pragma unroll 4
    for (int64_t it = (int64_t)blockIdx.x * kQuadsPerBlock + (threadIdx.x >> 2); it < items;
         it += (int64_t)gridDim.x * kQuadsPerBlock) {
        float v[4 * R];
        load_item<B>(xs, it * I, E, t, v);
#pragma unroll
        for (int r = 0; r < 4 * R; ++r) mx = fmaxf(mx, fabsf(v[r]));
        fwht_item<B>(v, t);
#pragma unroll
        for (int r = 0; r < 4 * R; ++r) mh = fmaxf(mh, fabsf(v[r]));
    }
    mx = wave_max(mx);
    mh = wave_max(mh);
    __shared__ float red[2][kThreads / 64];
    if ((threadIdx.x & 63) == 0) {
        red[0][threadIdx.x >> 6] = mx;
        red[1][threadIdx.x >> 6] = mh;
    }
    __syncthreads();
    if (threadIdx.x < 2) {
        float b = red[threadIdx.x][0];
#pragma unroll
        for (int w = 1; w < kThreads / 64; ++w) b = fmaxf(b, red[threadIdx.x][w]);
        atomic_max_nonneg(amax + (threadIdx.x ? gridDim.y : 0) + k, b);
    }
}

// Channels not a multiple of the block (or a ragged sample): one thread per
// (pixel, block), zero channels past C, the same ascending-bit butterfly in
// registers.
template <int B>
__global__ void __launch_bounds__(kThreads) range_pad_kernel(const float *__restrict__ x, int64_t P, int C,
                                                             float *__restrict__ amax) {
    const int k = blockIdx.y;
    const float *xs = x + (int64_t)k * P * C;
    const int nblk = (C + B - 1) / B;
    float mx = 0.0f, mh = 0.0f;
    for (int64_t u = (int64_t)blockIdx.x * kThreads + threadIdx.x; u < P * nblk; u += (int64_t)gridDim.x * kThreads) {
        const int64_t px = u / nblk;
        const int c0 = (int)(u - px * nblk) * B;
        float v[B];
#pragma unroll
        for (int j = 0; j < B; ++j) {
            v[j] = c0 + j < C ? xs[px * C + c0 + j] : 0.0f;
            mx = fmaxf(mx, fabsf(v[j]));
        }
#pragma unroll
        for (int h = 1; h < B; h <<= 1)
#pragma unroll
            for (int j = 0; j < B; ++j) {
                if (j & h) continue;
                const float a = v[j], c = v[j + h];
                v[j] = a + c;
                v[j + h] = a - c;
            }
#pragma unroll
        for (int j = 0; j < B; ++j) mh = fmaxf(mh, fabsf(v[j]));
    }
    mx = wave_max(mx);
    mh = wave_max(mh);
    __shared__ float red[2][kThreads / 64];
    if ((threadIdx.x & 63) == 0) {
        red[0][threadIdx.x >> 6] = mx;
        red[1][threadIdx.x >> 6] = mh;
    }
    __syncthreads();
    if (threadIdx.x < 2) {
        float b = red[threadIdx.x][0];
#pragma unroll
        for (int w = 1; w < kThreads / 64; ++w) b = fmaxf(b, red[threadIdx.x][w]);
        atomic_max_nonneg(amax + (threadIdx.x ? gridDim.y : 0) + k, b);
    }
}

// The indicator of each sample: max|S|^2 > b max|x|^2, exact in fp64 (the
// orthonormal transform is S / sqrt(b)); the expanding samples are counted.
__global__ void expansion_flags_kernel(const float *__restrict__ amax, int n, int b, int32_t *flags,
                                       int32_t *count) {
    const int k = blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= n) return;
    const double mx = amax[k], mh = amax[n + k];
    const int f = mh * mh > (double)b * (mx * mx);
    if (flags) flags[k] = f;
    if (count && f) atomicAdd(count, 1);
}

// Elementwise path for b <= 2 when E is not a multiple of 4 (float4 alignment
// of every sample cannot be assumed).  Element pairs never straddle a pixel
// because c % b == 0.
template <int B, bool QUANT>
__global__ void __launch_bounds__(kThreads) scalar_kernel(const float *__restrict__ x, int64_t E,
                                                          float *__restrict__ absmax,
                                                          int8_t *__restrict__ xq,
                                                          float *__restrict__ act_scale) {
    const int n = blockIdx.y;
    const float *xs = x + (int64_t)n * E;
    float s = 1.0f;
    if constexpr (QUANT) {
        s = act_scale_from_absmax(absmax[n]);
        if (blockIdx.x == 0 && threadIdx.x == 0) act_scale[n] = s;
    }
    float m = 0.0f;
    const int64_t groups = E / B;
    for (int64_t g = (int64_t)blockIdx.x * kThreads + threadIdx.x; g < groups;
         g += (int64_t)gridDim.x * kThreads) {
        float v[B];
#pragma unroll
        for (int j = 0; j < B; ++j) v[j] = xs[g * B + j];
        if constexpr (B == 2) {
            const float a = v[0], c = v[1];
            v[0] = a + c;
            v[1] = a - c;
        }
#pragma unroll
        for (int j = 0; j < B; ++j) {
            if constexpr (QUANT) xq[(int64_t)n * E + g * B + j] = (int8_t)(int)rintf(clamp127(v[j] / s));
            else m = fmaxf(m, fabsf(v[j]));
        }
    }
    if constexpr (!QUANT) {
        m = wave_max(m);
        if ((threadIdx.x & 63) == 0) atomic_max_nonneg(absmax + n, m);
    }
}

// Blocks per sample: enough for the work, at most `total` over the whole batch.
// Blocks of the quantization kernels over the whole batch (measured on the
// 805 M-element layer-2-shaped tensor: 16384 -> 32768 blocks 801 -> 782 us,
// 65536 no faster; on the 201 M-element one, blocks of 64, single read:
// 32768 -> 65536 blocks 175 -> 167 us NHWC, 178 -> 175 us chunk-major).
#ifndef HATQ_QUANT_GRID
#define HATQ_QUANT_GRID 65536
#endif
// The absmax kernels end in one atomic per block on one of the sample's
// kAbsSlots slots.
#ifndef HATQ_ABSMAX_GRID
#define HATQ_ABSMAX_GRID 4096
#endif
int grid_x(int64_t work_units, int per_block, int n, int total = HATQ_QUANT_GRID) {
    int64_t want = (work_units + per_block - 1) / per_block;
    int64_t cap = (total + n - 1) / n;
    if (cap < 1) cap = 1;
    if (want > cap) want = cap;
    return (int)(want < 1 ? 1 : want);
}

template <int B>
hipError_t launch_vector(const float *x, int n, int64_t E, const float *absmax_in, float *ws_absmax,
                         int8_t *xq, float *act_scale, hipStream_t st, int c64 = 0) {
    constexpr int I = ItemShape<B>::I;
    const int64_t items = (E + I - 1) / I;
    const float *A = absmax_in;
    if (!A) {
        fill_u32_kernel<<<1, 256, 0, st>>>(reinterpret_cast<uint32_t *>(ws_absmax), n * kAbsSlots, 0u);
        if constexpr (B == 1) {
            // sixteen float4 per thread
            const dim3 grid(grid_x(E / 4, kThreads * 16, n, HATQ_ABSMAX_GRID), n);
            absmax_flat_kernel<<<grid, kThreads, 0, st>>>(x, E, ws_absmax);
        } else {
            const dim3 grid(grid_x(items, kQuadsPerBlock, n, HATQ_ABSMAX_GRID), n);
            absmax_kernel<B><<<grid, kThreads, 0, st>>>(x, E, ws_absmax);
        }
        A = ws_absmax;
    }
    const int slots = absmax_in ? 1 : kAbsSlots;
    dim3 grid(grid_x(items, kQuadsPerBlock * QuantUnroll<B>::UN, n), n);
    quant_kernel<B><<<grid, kThreads, 0, st>>>(x, E, A, xq, act_scale, c64, slots);
    return hipGetLastError();
}

template <int B>
hipError_t launch_scalar(const float *x, int n, int64_t E, const float *absmax_in, float *ws_absmax,
                         int8_t *xq, float *act_scale, hipStream_t st) {
    dim3 grid(grid_x(E / B, kThreads, n), n);
    const float *A = absmax_in;
    if (!A) {
        fill_u32_kernel<<<1, 256, 0, st>>>(reinterpret_cast<uint32_t *>(ws_absmax), n, 0u);
        scalar_kernel<B, false><<<dim3(grid_x(E / B, kThreads, n, 2048), n), kThreads, 0, st>>>(x, E, ws_absmax,
                                                                                              nullptr, nullptr);
        A = ws_absmax;
    }
    scalar_kernel<B, true><<<grid, kThreads, 0, st>>>(x, E, const_cast<float *>(A), xq, act_scale);
    return hipGetLastError();
}

template <int B>
hipError_t launch_range_b(const float *x, int n, int64_t P, int C, float *amax, hipStream_t st) {
    const int64_t E = P * C;
    if (C % B == 0 && E % 4 == 0) {
        constexpr int I = ItemShape<B>::I;
        const int64_t items = (E + I - 1) / I;
        range_kernel<B><<<dim3(grid_x(items, kQuadsPerBlock, n, 2048), n), kThreads, 0, st>>>(x, E, amax);
    } else if constexpr (kron_q(B) == 0) {
        const int64_t units = P * ((C + B - 1) / B);
        range_pad_kernel<B><<<dim3(grid_x(units, kThreads, n, 2048), n), kThreads, 0, st>>>(x, P, C, amax);
    } else {
        return hipErrorInvalidValue;   // Kronecker orders: whole blocks only
    }
    return hipGetLastError();
}

template <int B>
hipError_t launch_affine_b(const float *x, int n, int64_t E, float *ws, int8_t *xq, float *act_scale,
                           int32_t *act_zero, hipStream_t st) {
    constexpr int I = ItemShape<B>::I;
    const int64_t items = (E + I - 1) / I;
    fill_u32_kernel<<<1, 256, 0, st>>>(reinterpret_cast<uint32_t *>(ws), 2 * n, 0u);
    minmax_kernel<B><<<dim3(grid_x(items, kQuadsPerBlock, n, 2048), n), kThreads, 0, st>>>(x, E, ws);
    quant_affine_kernel<B><<<dim3(grid_x(items, kQuadsPerBlock, n), n), kThreads, 0, st>>>(x, E, ws, xq, act_scale,
                                                                                          act_zero);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_act_quant_affine(const float *x, int n, int64_t E, int hblock, float *ws, int8_t *xq,
                                   float *act_scale, int32_t *act_zero, hipStream_t st) {
    if (E % 4 != 0) return hipErrorInvalidValue;
    switch (hblock) {
        case 1: return launch_affine_b<1>(x, n, E, ws, xq, act_scale, act_zero, st);
        case 2: return launch_affine_b<2>(x, n, E, ws, xq, act_scale, act_zero, st);
        case 4: return launch_affine_b<4>(x, n, E, ws, xq, act_scale, act_zero, st);
        case 8: return launch_affine_b<8>(x, n, E, ws, xq, act_scale, act_zero, st);
        case 16: return launch_affine_b<16>(x, n, E, ws, xq, act_scale, act_zero, st);
        case 32: return launch_affine_b<32>(x, n, E, ws, xq, act_scale, act_zero, st);
        case 64: return launch_affine_b<64>(x, n, E, ws, xq, act_scale, act_zero, st);
        case 128: return launch_affine_b<128>(x, n, E, ws, xq, act_scale, act_zero, st);
        case 192: return launch_affine_b<192>(x, n, E, ws, xq, act_scale, act_zero, st);
        case 320: return launch_affine_b<320>(x, n, E, ws, xq, act_scale, act_zero, st);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_range_expansion(const float *x, int n, int64_t P, int C, int hblock, float *amax, int32_t *flags,
                                  int32_t *count, hipStream_t st) {
    fill_u32_kernel<<<1, 256, 0, st>>>(reinterpret_cast<uint32_t *>(amax), 2 * n, 0u);
    hipError_t e;
    switch (hblock) {
        case 1: e = launch_range_b<1>(x, n, P, C, amax, st); break;
        case 2: e = launch_range_b<2>(x, n, P, C, amax, st); break;
        case 4: e = launch_range_b<4>(x, n, P, C, amax, st); break;
        case 8: e = launch_range_b<8>(x, n, P, C, amax, st); break;
        case 16: e = launch_range_b<16>(x, n, P, C, amax, st); break;
        case 32: e = launch_range_b<32>(x, n, P, C, amax, st); break;
        case 64: e = launch_range_b<64>(x, n, P, C, amax, st); break;
        case 128: e = launch_range_b<128>(x, n, P, C, amax, st); break;
        case 192: e = launch_range_b<192>(x, n, P, C, amax, st); break;
        case 320: e = launch_range_b<320>(x, n, P, C, amax, st); break;
        default: return hipErrorInvalidValue;
    }
    if (e != hipSuccess) return e;
    expansion_flags_kernel<<<(n + 255) / 256, 256, 0, st>>>(amax, n, hblock, flags, count);
    return hipGetLastError();
}

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
float *g_scratch[kMaxDevices] = {};

// The current device's copy of `scratch`, looked up on the first call on that
// device (with it current) and kept.
hipError_t scratch_absmax(float **out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        g_scratch[dev] = static_cast<float *>(p);
    }
    *out = g_scratch[dev];
    return hipSuccess;
}

}  // namespace

hipError_t launch_act_quant_noalloc(const float *x, int n, int64_t E, int hblock, int8_t *xq, float *act_scale,
                                    hipStream_t st) {
    if (n <= 0 || n > kNoAllocMaxSamples) return hipErrorInvalidValue;
    float *ws = nullptr;
    const hipError_t e = scratch_absmax(&ws);
    if (e != hipSuccess) return e;
    // the two-pass path clears the n * kAbsSlots slots with a fill kernel
    // before its atomics
    return launch_act_quant(x, n, E, hblock, nullptr, ws, xq, act_scale, st);
}

hipError_t launch_act_quant(const float *x, int n, int64_t E, int hblock, const float *absmax_in,
                            float *ws_absmax, int8_t *xq, float *act_scale, hipStream_t st, int c64) {
    if (c64 > 0) {
        // items of 64 channels, one chunk each
        if (c64 % 64 != 0 || E % c64 != 0) return hipErrorInvalidValue;
        switch (hblock) {
            case 1: return launch_vector<1>(x, n, E, absmax_in, ws_absmax, xq, act_scale, st, c64);
            case 2: return launch_vector<2>(x, n, E, absmax_in, ws_absmax, xq, act_scale, st, c64);
            case 4: return launch_vector<4>(x, n, E, absmax_in, ws_absmax, xq, act_scale, st, c64);
            case 8: return launch_vector<8>(x, n, E, absmax_in, ws_absmax, xq, act_scale, st, c64);
            case 16: return launch_vector<16>(x, n, E, absmax_in, ws_absmax, xq, act_scale, st, c64);
            case 32: return launch_vector<32>(x, n, E, absmax_in, ws_absmax, xq, act_scale, st, c64);
            case 64: return launch_vector<64>(x, n, E, absmax_in, ws_absmax, xq, act_scale, st, c64);
            default: return hipErrorInvalidValue;
        }
    }
    if (E % 4 != 0) {
        if (hblock == 1) return launch_scalar<1>(x, n, E, absmax_in, ws_absmax, xq, act_scale, st);
        return launch_scalar<2>(x, n, E, absmax_in, ws_absmax, xq, act_scale, st);
    }
    switch (hblock) {
        case 1: return launch_vector<1>(x, n, E, absmax_in, ws_absmax, xq, act_scale, st);
        case 2: return launch_vector<2>(x, n, E, absmax_in, ws_absmax, xq, act_scale, st);
        case 4: return launch_vector<4>(x, n, E, absmax_in, ws_absmax, xq, act_scale, st);
        case 8: return launch_vector<8>(x, n, E, absmax_in, ws_absmax, xq, act_scale, st);
        case 16: return launch_vector<16>(x, n, E, absmax_in, ws_absmax, xq, act_scale, st);
        case 32: return launch_vector<32>(x, n, E, absmax_in, ws_absmax, xq, act_scale, st);
        case 64: return launch_vector<64>(x, n, E, absmax_in, ws_absmax, xq, act_scale, st);
        case 128: return launch_vector<128>(x, n, E, absmax_in, ws_absmax, xq, act_scale, st);
        case 192: return launch_vector<192>(x, n, E, absmax_in, ws_absmax, xq, act_scale, st);
        case 320: return launch_vector<320>(x, n, E, absmax_in, ws_absmax, xq, act_scale, st);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace hatq
