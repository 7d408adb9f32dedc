// INT8 implicit-GEMM convolution with INT32 accumulation and fused epilogue
// (steps a5-a6) on gfx950 MFMA (v_mfma_i32_16x16x64_i8).
//
// GEMM view (Eq. linear_operator): rows = output points, columns = output
// channels, contraction d = tap * cin_p + ci.  One K-step is 64 contraction
// values: 64 channels of one tap (regular path) or 64 consecutive d's of a
// small-cin layer (cin <= 8, d gathered byte by byte).
//
// Block tile BM x BN, 4 waves stacked along M (each wave TM = BM/4 rows by all
// BN columns, so a wave owns whole 64-channel blocks for the WH restore).
// Per K-step the A tile (BM rows x 64 B, an on-the-fly im2col) and the B tile
// (BN columns x 64 B of the prepared weights) go global -> registers -> LDS,
// double buffered with one barrier per K-step; the next K-step's global loads
// are in flight while the current one runs on MFMA.  LDS rows are 64 B with the
// four 16-B chunks XOR-swizzled by the row index so the 16-row fragment reads
// spread over all banks.
//
// Epilogue (accumulators in registers, MFMA C layout: lane l, register r holds
// row 4*(l/16) + r, column l % 16 of each 16 x 16 tile):
//   I32: raw accumulators.
//   DH : y = fma(float(acc), fl(s_x * s_w,c) * (1/b), bias_c).
//   WH : z = fma(float(acc), fl(s_x * s_w,c), b~_c), then the b-point FWHT along
//        the channels of each 64-block (lane bits 0-3 by DPP, tile index bits 4+
//        in registers), times 1/b, truncated to cout.
//   next_absmax: max |B_next y| per sample with the same ascending-bit butterfly
//        as the activation kernels, so it equals what they would compute.
#include "hatq_device.h"
#include "hatq_launch.h"

namespace hatq {
namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ int swz(int row) { return ((row >> 1) ^ (row >> 3)) & 3; }

// Butterfly along the column-tile index (register) dimension of a [FN][4] array.
template <int S, int FN>
__device__ __forceinline__ void tile_stage(float (&v)[FN][4]) {
#pragma unroll
    for (int f = 0; f < FN; ++f) {
        if (f & S) continue;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const float a = v[f][r], c = v[f + S][r];
            v[f][r] = a + c;
            v[f + S][r] = a - c;
        }
    }
}

template <int MASK, int FN>
__device__ __forceinline__ void lane_stage(float (&v)[FN][4], float coef) {
#pragma unroll
    for (int f = 0; f < FN; ++f)
#pragma unroll
        for (int r = 0; r < 4; ++r) v[f][r] = __builtin_fmaf(coef, lane_xor<MASK>(v[f][r]), v[f][r]);
}

// In-place FWHT of order b along channels (column n = 16*f + lane%16 inside a
// block), ascending bit order.  Returns the per-lane sign sigma of the result.
template <int FN>
__device__ __forceinline__ float fwht_cols(float (&v)[FN][4], int b, int lane) {
    float sigma = 1.0f;
    const int l = lane & 15;
    if (b >= 2) { const float c = (l & 1) ? -1.f : 1.f; lane_stage<1>(v, c); sigma *= c; }
    if (b >= 4) { const float c = (l & 2) ? -1.f : 1.f; lane_stage<2>(v, c); sigma *= c; }
    if (b >= 8) { const float c = (l & 4) ? -1.f : 1.f; lane_stage<4>(v, c); sigma *= c; }
    if (b >= 16) { const float c = (l & 8) ? -1.f : 1.f; lane_stage<8>(v, c); sigma *= c; }
    if constexpr (FN % 2 == 0) if (b >= 32) tile_stage<1>(v);
    if constexpr (FN % 4 == 0) if (b >= 64) tile_stage<2>(v);
    if constexpr (FN % 8 == 0) if (b >= 128) tile_stage<4>(v);
    return sigma;
}

struct RowInfo {
    int64_t out_off;   // output pixel index (n, oh, ow) flattened, or -1
    int nb;
};

__device__ __forceinline__ RowInfo row_info(const ConvArgs &a, int64_t R) {
    RowInfo ri;
    if (R >= a.M) { ri.out_off = -1; ri.nb = 0; return ri; }
    const int64_t ghw = (int64_t)a.gh * a.gw;
    const int nb = (int)(R / ghw);
    const int64_t rem = R - (int64_t)nb * ghw;
    const int gi = (int)(rem / a.gw), gj = (int)(rem - (int64_t)gi * a.gw);
    const int oh = gi * a.so + a.boh, ow = gj * a.so + a.bow;
    ri.nb = nb;
    ri.out_off = ((int64_t)nb * a.ho + oh) * a.wo + ow;
    return ri;
}

template <int BM, int BN, int CIN_SMALL>
__global__ void __launch_bounds__(kThreads, 1) conv_kernel(const ConvArgs a) {
    constexpr int TM = BM / 4;
    constexpr int FM = TM / 16;
    constexpr int FN = BN / 16;
    constexpr int A_PIECES = BM * 4 / kThreads;
    constexpr int B_PIECES = BN * 4 / kThreads;
    constexpr int BUF = (BM + BN) * 64;
    static_assert(BM * 4 % kThreads == 0 && BN * 4 % kThreads == 0, "tile");
    __shared__ __attribute__((aligned(16))) int8_t lds[2 * BUF];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;

    // XCD-aware tile order: blocks bid, bid+8, ... run on one XCD; give each
    // XCD a contiguous range of tiles so neighbouring tiles share its L2.
    const int nt = gridDim.x;
    const int bid = blockIdx.x;
    const int xcd = bid & 7, q = nt >> 3, rmd = nt & 7;
    const int logical = xcd * q + (xcd < rmd ? xcd : rmd) + (bid >> 3);
    const int tile_m = logical / a.tiles_n;
    const int tile_n = logical - tile_m * a.tiles_n;
    const int64_t m0 = (int64_t)tile_m * BM;
    const int n0 = tile_n * BN;

    // ---- per-thread A-load rows ----
    const int g = tid & 3;
    const int8_t *a_base[A_PIECES];
    int a_ih0[A_PIECES], a_iw0[A_PIECES];
#pragma unroll
    for (int p = 0; p < A_PIECES; ++p) {
        const int m = (tid >> 2) + 64 * p;
        const int64_t R = m0 + m;
        if (R < a.M) {
            const int64_t ghw = (int64_t)a.gh * a.gw;
            const int nb = (int)(R / ghw);
            const int64_t rem = R - (int64_t)nb * ghw;
            const int gi = (int)(rem / a.gw), gj = (int)(rem - (int64_t)gi * a.gw);
            a_ih0[p] = gi * a.sa + a.bah;
            a_iw0[p] = gj * a.sa + a.baw;
            a_base[p] = a.xq + (int64_t)nb * a.h * a.w * a.cin_p;
        } else {
            a_ih0[p] = -(1 << 28);   // every tap out of range
            a_iw0[p] = 0;
            a_base[p] = a.xq;
        }
    }

    // Small-cin path: per contraction index d, the tap offset, channel and the
    // byte offset relative to the anchor pixel.
    __shared__ int s_lut_off[CIN_SMALL ? 128 : 1];
    __shared__ int8_t s_lut_dh[CIN_SMALL ? 128 : 1], s_lut_dw[CIN_SMALL ? 128 : 1];
    if constexpr (CIN_SMALL > 0) {
        if (tid < 128) {
            const int d = tid;
            if (d < a.k_total) {
                const int t = d / CIN_SMALL, ci = d - t * CIN_SMALL;
                s_lut_dh[d] = a.dh[t];
                s_lut_dw[d] = a.dw[t];
                s_lut_off[d] = (a.dh[t] * a.w + a.dw[t]) * CIN_SMALL + ci;
            } else {
                // past the contraction: read the (bounds-checked) anchor pixel;
                // the prepared weights are zero there, so it contributes 0
                s_lut_dh[d] = 0;
                s_lut_dw[d] = 0;
                s_lut_off[d] = 0;
            }
        }
        __syncthreads();
    }

    v4i ra[A_PIECES], rb[B_PIECES];
    const int cin_p = a.cin_p;
    const int nchunks = CIN_SMALL ? 1 : cin_p >> 6;

    auto global_load = [&](int ks) {
        if constexpr (CIN_SMALL == 0) {
            const int tap = ks / nchunks;
            const int chunk = ks - tap * nchunks;
            const int dh = a.dh[tap], dw = a.dw[tap];
            const int64_t coff = (int64_t)(dh * a.w + dw) * cin_p + chunk * 64 + g * 16;
#pragma unroll
            for (int p = 0; p < A_PIECES; ++p) {
                const int ih = a_ih0[p] + dh, iw = a_iw0[p] + dw;
                v4i v = {0, 0, 0, 0};
                if ((unsigned)ih < (unsigned)a.h && (unsigned)iw < (unsigned)a.w)
                    v = *reinterpret_cast<const v4i *>(a_base[p] + ((int64_t)a_ih0[p] * a.w + a_iw0[p]) * cin_p + coff);
                ra[p] = v;
            }
            const int64_t woff = (int64_t)a.wtap[tap] * cin_p + chunk * 64 + g * 16;
#pragma unroll
            for (int p = 0; p < B_PIECES; ++p) {
                const int nn = (tid >> 2) + 64 * p;
                rb[p] = *reinterpret_cast<const v4i *>(a.wq + (int64_t)(n0 + nn) * a.k_stride + woff);
            }
        } else {
            const int d0 = ks * 64 + g * 16;
#pragma unroll
            for (int p = 0; p < A_PIECES; ++p) {
                uint32_t wv[4];
                const int64_t pix = ((int64_t)a_ih0[p] * a.w + a_iw0[p]) * CIN_SMALL;
#pragma unroll
                for (int e4 = 0; e4 < 4; ++e4) {
                    uint32_t word = 0;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int d = d0 + 4 * e4 + e;
                        const int ih = a_ih0[p] + s_lut_dh[d], iw = a_iw0[p] + s_lut_dw[d];
                        uint32_t byte = 0;
                        if ((unsigned)ih < (unsigned)a.h && (unsigned)iw < (unsigned)a.w)
                            byte = (uint8_t)a_base[p][pix + s_lut_off[d]];
                        word |= byte << (8 * e);
                    }
                    wv[e4] = word;
                }
                ra[p] = v4i{(int)wv[0], (int)wv[1], (int)wv[2], (int)wv[3]};
            }
#pragma unroll
            for (int p = 0; p < B_PIECES; ++p) {
                const int nn = (tid >> 2) + 64 * p;
                rb[p] = *reinterpret_cast<const v4i *>(a.wq + (int64_t)(n0 + nn) * a.k_stride + d0);
            }
        }
    };

    auto lds_store = [&](int buf) {
        int8_t *base = lds + buf * BUF;
#pragma unroll
        for (int p = 0; p < A_PIECES; ++p) {
            const int m = (tid >> 2) + 64 * p;
            *reinterpret_cast<v4i *>(base + m * 64 + 16 * (g ^ swz(m))) = ra[p];
        }
#pragma unroll
        for (int p = 0; p < B_PIECES; ++p) {
            const int nn = (tid >> 2) + 64 * p;
            *reinterpret_cast<v4i *>(base + BM * 64 + nn * 64 + 16 * (g ^ swz(nn))) = rb[p];
        }
    };

    v4i acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = v4i{0, 0, 0, 0};

    const int nks = a.nksteps;
    global_load(0);
    lds_store(0);
    __syncthreads();

    const int fr = lane & 15, fg = lane >> 4;
    for (int ks = 0; ks < nks; ++ks) {
        const int buf = ks & 1;
        if (ks + 1 < nks) global_load(ks + 1);
        const int8_t *base = lds + buf * BUF;
        v4i fa[FM], fb[FN];
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            const int m = wave * TM + 16 * i + fr;
            fa[i] = *reinterpret_cast<const v4i *>(base + m * 64 + 16 * (fg ^ swz(m)));
        }
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const int nn = 16 * j + fr;
            fb[j] = *reinterpret_cast<const v4i *>(base + BM * 64 + nn * 64 + 16 * (fg ^ swz(nn)));
        }
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[i], fb[j], acc[i][j], 0, 0, 0);
        if (ks + 1 < nks) lds_store(buf ^ 1);
        __syncthreads();
    }

    // ---------------------------- epilogue ----------------------------------
    const int col_l = lane & 15;
    if (a.mode == 0) {
        int32_t *y = reinterpret_cast<int32_t *>(a.y);
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const RowInfo ri = row_info(a, m0 + wave * TM + 16 * i + 4 * fg + r);
                if (ri.out_off < 0) continue;
                int32_t *yr = y + ri.out_off * a.cout_pad + n0 + col_l;
#pragma unroll
                for (int j = 0; j < FN; ++j) yr[16 * j] = acc[i][j][r];
            }
        return;
    }

    float *y = reinterpret_cast<float *>(a.y);
    const float inv_b = 1.0f / (float)a.hblock;
    // the tile's rows all belong to one sample?
    const int64_t last_row = (m0 + BM <= a.M ? m0 + BM : a.M) - 1;
    const int64_t ghw = (int64_t)a.gh * a.gw;
    const bool one_sample = (m0 / ghw) == (last_row / ghw);
    float wave_m = 0.0f;

#pragma unroll
    for (int i = 0; i < FM; ++i) {
        RowInfo ri[4];
        float sxr[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            ri[r] = row_info(a, m0 + wave * TM + 16 * i + 4 * fg + r);
            sxr[r] = a.sx[ri[r].nb];
        }
        float v[FN][4];
        if (a.form == 0) {
#pragma unroll
            for (int j = 0; j < FN; ++j) {
                const int c = n0 + 16 * j + col_l;
                const float sw = a.w_scale[c], bi = a.bias[c];
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    v[j][r] = __builtin_fmaf((float)acc[i][j][r], (sxr[r] * sw) * inv_b, bi);
            }
        } else {
#pragma unroll
            for (int j = 0; j < FN; ++j) {
                const int c = n0 + 16 * j + col_l;
                const float sw = a.w_scale[c], bi = a.bias[c];
#pragma unroll
                for (int r = 0; r < 4; ++r) v[j][r] = __builtin_fmaf((float)acc[i][j][r], sxr[r] * sw, bi);
            }
            const float sg = fwht_cols<FN>(v, a.hblock, lane) * inv_b;
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int r = 0; r < 4; ++r) v[j][r] *= sg;
        }
        // store y (original basis), columns < cout
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            if (ri[r].out_off < 0) continue;
            float *yr = y + ri[r].out_off * a.cout + n0 + col_l;
#pragma unroll
            for (int j = 0; j < FN; ++j)
                if (n0 + 16 * j + col_l < a.cout) yr[16 * j] = v[j][r];
        }
        if (a.next_hblock > 0 && a.next_absmax) {
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    if (n0 + 16 * j + col_l >= a.cout || ri[r].out_off < 0) v[j][r] = 0.0f;
            if (a.next_hblock > 1) fwht_cols<FN>(v, a.next_hblock, lane);
            if (one_sample) {
#pragma unroll
                for (int j = 0; j < FN; ++j)
#pragma unroll
                    for (int r = 0; r < 4; ++r) wave_m = fmaxf(wave_m, fabsf(v[j][r]));
            } else {
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    float rm = 0.0f;
#pragma unroll
                    for (int j = 0; j < FN; ++j) rm = fmaxf(rm, fabsf(v[j][r]));
                    if (ri[r].out_off >= 0) atomic_max_nonneg(a.next_absmax + ri[r].nb, rm);
                }
            }
        }
    }
    if (a.next_hblock > 0 && a.next_absmax && one_sample) {
        wave_m = wave_max(wave_m);
        if (lane == 0) atomic_max_nonneg(a.next_absmax + m0 / ghw, wave_m);
    }
}

template <int BM, int BN, int CS>
hipError_t launch_tile(const ConvArgs &a, hipStream_t st) {
    ConvArgs b = a;
    b.tiles_m = (int)((a.M + BM - 1) / BM);
    b.tiles_n = a.cout_pad / BN;
    const int64_t tiles = (int64_t)b.tiles_m * b.tiles_n;
    if (tiles <= 0 || tiles > (int64_t)1 << 31) return hipErrorInvalidValue;
    conv_kernel<BM, BN, CS><<<(unsigned)tiles, kThreads, 0, st>>>(b);
    return hipGetLastError();
}

template <int CS>
hipError_t launch_by_n(const ConvArgs &a, hipStream_t st) {
    switch (a.cout_pad) {
        case 64: return launch_tile<256, 64, CS>(a, st);
        case 128: return launch_tile<256, 128, CS>(a, st);
        case 192: return launch_tile<256, 192, CS>(a, st);
        case 256: return launch_tile<128, 256, CS>(a, st);
        case 320: return launch_tile<128, 320, CS>(a, st);
        default: break;
    }
    if (a.cout_pad % 64 == 0 && (a.form == 0 || a.hblock <= 64) && a.next_hblock <= 64)
        return launch_tile<256, 64, CS>(a, st);
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_conv(const ConvArgs &a, bool clear_next, hipStream_t st) {
    if (clear_next && a.next_absmax && a.next_hblock > 0)
        fill_u32_kernel<<<1, 256, 0, st>>>(reinterpret_cast<uint32_t *>(a.next_absmax), a.n, 0u);
    switch (a.cin_p <= 8 ? a.cin_p : 0) {
        case 0: return launch_by_n<0>(a, st);
        case 1: return launch_by_n<1>(a, st);
        case 2: return launch_by_n<2>(a, st);
        case 3: return launch_by_n<3>(a, st);
        case 4: return launch_by_n<4>(a, st);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace hatq
