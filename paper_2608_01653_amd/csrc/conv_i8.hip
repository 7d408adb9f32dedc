// INT8 implicit-GEMM convolution with INT32 accumulation and fused epilogue
// (steps a5-a6) on gfx950 MFMA (v_mfma_i32_16x16x64_i8).
//
// GEMM view (Eq. linear_operator): rows = output points (pixels), columns =
// output channels, contraction d = tap * cin_p + ci.  One K-step is 64
// contraction values: 64 channels of one tap (regular path) or 64 consecutive
// d's of a small-cin layer (cin <= 4, gathered byte by byte).
//
// Block tile BM x BN, 4 waves stacked along M: each wave owns TM = BM/4 pixels
// by all BN channels.  The MFMA takes the weight fragment as its first operand,
// so the accumulator layout is channels x pixels: lane l, register r of tile
// (i, j) holds channel 16*j + 4*(l/16) + r of pixel 16*i + l%16, i.e. four
// consecutive channels of one pixel.
//
// Epilogue, per 16-pixel group, through a wave-private LDS staging area:
//   1. dequantize (DH: y = fma(float(acc), fl(s_x*s_w,c)*(1/b), bias_c);
//      WH: z = fma(float(acc), fl(s_x*s_w,c), b~_c); I32: raw) and write 16 B
//      per lane into staged rows of BN floats (float4 columns XOR-swizzled by
//      the row so both access patterns below are bank-conflict free);
//   2. re-read in the quad layout of the activation kernels (one quad per
//      64-channel block of one pixel) for the WH output-basis restore (b-point
//      FWHT, times 1/b) and for the next layer's per-sample max |B_next y|, with
//      the very butterfly the activation kernels use, so the max equals what
//      they would compute from the stored y;
//   3. store every staged row as one contiguous run of 16-B lanes.
#include <utility>

#include "hatq_device.h"
#include "hatq_launch.h"

namespace hatq {
namespace {

constexpr int kThreads = 256;

// 16-B chunk swizzle of a 64-B LDS operand row (A and B tiles).
__device__ __forceinline__ int swz(int row) { return ((row >> 1) ^ (row >> 3)) & 3; }

// float4-column swizzle of a staged epilogue row: a bijection of the low four
// bits of the column, different for each of 16 consecutive rows.
__device__ __forceinline__ int stg_swz(int row) { return ((row & 3) << 2) | ((row >> 2) & 3); }

// Quad-layout butterfly of runtime order b <= 64 (wave-uniform branches): the
// same stages in the same order as fwht_item<b>, hence the same fp32 results.
__device__ __forceinline__ float fwht16(float (&v)[16], int b, int qt) {
    float sigma = 1.0f;
    if (b >= 2) reg_stage<1>(v);
    if (b >= 4) reg_stage<2>(v);
    if (b >= 8) {
        const float c = (qt & 1) ? -1.0f : 1.0f;
        cross_stage<1>(v, c);
        sigma *= c;
    }
    if (b >= 16) {
        const float c = (qt & 2) ? -1.0f : 1.0f;
        cross_stage<2>(v, c);
        sigma *= c;
    }
    if (b >= 32) reg_stage<4>(v);
    if (b >= 64) reg_stage<8>(v);
    return sigma;
}

// A block's tile: sample nb, first grid point (gi0, gj0); local row m is the
// point (gi0 + m / TW, gj0 + m % TW).  Tiles never straddle samples.
struct Tile {
    int nb, gi0, gj0, n0;
};

__device__ __forceinline__ Tile block_tile(const ConvArgs &a, int logical, int TH, int TW, int BN) {
    Tile t;
    const int tile_m = logical / a.tiles_n;
    t.n0 = (logical - tile_m * a.tiles_n) * BN;
    const int per = a.tiles_h * a.tiles_w;
    t.nb = tile_m / per;
    const int rem = tile_m - t.nb * per;
    const int th = rem / a.tiles_w;
    t.gi0 = th * TH;
    t.gj0 = (rem - th * a.tiles_w) * TW;
    return t;
}

// Output pixel index of grid point (nb, gi, gj).
__device__ __forceinline__ int64_t out_pixel(const ConvArgs &a, int nb, int gi, int gj) {
    return ((int64_t)nb * a.ho + gi * a.so + a.boh) * a.wo + gj * a.so + a.bow;
}

struct EpiCtx {
    Tile t;
    int lane, ycols, ncols;
    bool f32, wh, want_abs;
    float inv_b;
    const float *col_t;   // LDS: per column, fl(s_x*s_w,c) (WH) or fl(fl(s_x*s_w,c)/b) (DH)
    const float *col_b;   // LDS: per column bias
};

// One 16-point group (local rows row0 + 16*I ... + 15: one tile row segment,
// since 16 divides TW) of a wave's accumulator tile.
template <int I, int TW, int FM, int FN>
__device__ __forceinline__ void epilogue_group(const ConvArgs &a, const EpiCtx &e, const v4i (&acc)[FM][FN],
                                               int row0, float *stg, float &wave_m) {
    constexpr int BN = 16 * FN;
    constexpr int NBLK = BN / 64;
    static_assert(TW % 16 == 0, "a 16-point group must lie in one tile row");
    const int lane = e.lane;
    const int pl = lane & 15, cg = lane >> 4;
    const int qrow = lane >> 2, qt = lane & 3;
    const int n0 = e.t.n0;
    const int m0 = row0 + 16 * I;                 // first local row of the group
    const int gi = e.t.gi0 + m0 / TW;             // its grid row (same for all 16)
    const int gj0 = e.t.gj0 + m0 % TW;            // grid column of row 0 of the group
    const bool row_ok = gi < a.gh;
    // 1. dequantize into the staged rows
    {
        float *srow = stg + pl * BN;
        const int sw_row = stg_swz(pl);
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const int cl = 16 * j + 4 * cg;   // column inside the tile
            float4 o;
            if (!e.f32) {
                o = make_float4(__int_as_float(acc[I][j][0]), __int_as_float(acc[I][j][1]),
                                __int_as_float(acc[I][j][2]), __int_as_float(acc[I][j][3]));
            } else {
                const float4 t4 = *reinterpret_cast<const float4 *>(e.col_t + cl);
                const float4 b4 = *reinterpret_cast<const float4 *>(e.col_b + cl);
                o.x = __builtin_fmaf((float)acc[I][j][0], t4.x, b4.x);
                o.y = __builtin_fmaf((float)acc[I][j][1], t4.y, b4.y);
                o.z = __builtin_fmaf((float)acc[I][j][2], t4.z, b4.z);
                o.w = __builtin_fmaf((float)acc[I][j][3], t4.w, b4.w);
            }
            const int q = 4 * j + cg;   // float4 column
            *reinterpret_cast<float4 *>(srow + 4 * (q ^ sw_row)) = o;
        }
    }
    // 2. WH restore and next-operand absmax in the quad layout (same wave: its
    //    LDS writes above are ordered before these reads)
    if (e.wh || e.want_abs) {
        const bool rvalid = row_ok && gj0 + qrow < a.gw;
        float *srow = stg + qrow * BN;
        const int sw_row = stg_swz(qrow);
        for (int k = 0; k < NBLK; ++k) {
            float v[16];
#pragma unroll
            for (int ii = 0; ii < 4; ++ii) {
                const int q = 16 * k + 4 * ii + qt;
                const float4 f = *reinterpret_cast<const float4 *>(srow + 4 * (q ^ sw_row));
                v[4 * ii] = f.x;
                v[4 * ii + 1] = f.y;
                v[4 * ii + 2] = f.z;
                v[4 * ii + 3] = f.w;
            }
            if (e.wh) {
                const float sg = fwht16(v, a.hblock, qt) * e.inv_b;
#pragma unroll
                for (int r = 0; r < 16; ++r) v[r] *= sg;
#pragma unroll
                for (int ii = 0; ii < 4; ++ii) {
                    const int q = 16 * k + 4 * ii + qt;
                    *reinterpret_cast<float4 *>(srow + 4 * (q ^ sw_row)) =
                        make_float4(v[4 * ii], v[4 * ii + 1], v[4 * ii + 2], v[4 * ii + 3]);
                }
            }
            if (e.want_abs) {
                // channels past cout and rows past M are not part of the next operand
#pragma unroll
                for (int ii = 0; ii < 4; ++ii)
#pragma unroll
                    for (int jj = 0; jj < 4; ++jj) {
                        const int ch = n0 + 64 * k + 16 * ii + 4 * qt + jj;
                        if (!rvalid || ch >= a.cout) v[4 * ii + jj] = 0.0f;
                    }
                fwht16(v, a.next_hblock, qt);
                float m = 0.0f;
#pragma unroll
                for (int r = 0; r < 16; ++r) m = fmaxf(m, fabsf(v[r]));
                wave_m = fmaxf(wave_m, m);
            }
        }
    }
    // 3. each staged row is one contiguous run of y
    if (!row_ok) return;
    const bool vec = (e.ycols & 3) == 0;
    float *y0 = reinterpret_cast<float *>(a.y) + out_pixel(a, e.t.nb, gi, gj0) * e.ycols + n0;
    const int64_t ystep = (int64_t)a.so * e.ycols;   // consecutive grid columns
    for (int r = 0; r < 16; ++r) {
        if (gj0 + r >= a.gw) break;
        float *yr = y0 + r * ystep;
        const float *srow = stg + r * BN;
        const int sw_row = stg_swz(r);
        if (vec) {
            for (int q = lane; 4 * q < e.ncols; q += 64)
                *reinterpret_cast<float4 *>(yr + 4 * q) =
                    *reinterpret_cast<const float4 *>(srow + 4 * (q ^ sw_row));
        } else {
            for (int c = lane; c < e.ncols; c += 64) yr[c] = srow[4 * ((c >> 2) ^ sw_row) + (c & 3)];
        }
    }
}

template <int TW, int FM, int FN, int... Is>
__device__ __forceinline__ void epilogue_groups(const ConvArgs &a, const EpiCtx &e, const v4i (&acc)[FM][FN],
                                                int row0, float *stg, float &wave_m,
                                                std::integer_sequence<int, Is...>) {
    (epilogue_group<Is, TW, FM, FN>(a, e, acc, row0, stg, wave_m), ...);
}

// Per-tile column factors of the dequantization (the tile is one sample, so
// s_x is uniform): col_t[c] = fl(s_x*s_w,c) for WH, fl(fl(s_x*s_w,c) * (1/b))
// for DH (exact power of two); col_b[c] = bias.  Written by the whole block.
template <int BN>
__device__ __forceinline__ void column_factors(const ConvArgs &a, const Tile &t, float *col_t, float *col_b) {
    const float sxv = a.sx[t.nb];
    const float f = a.form == 1 ? 1.0f : 1.0f / (float)a.hblock;
    for (int c = threadIdx.x; c < BN; c += kThreads) {
        col_t[c] = (sxv * a.w_scale[t.n0 + c]) * f;
        col_b[c] = a.bias[t.n0 + c];
    }
}

// row0: the wave's first local row in the tile.  col_t / col_b: LDS column
// factors (column_factors, followed by a block barrier).
template <int TW, int FM, int FN>
__device__ __forceinline__ void epilogue(const ConvArgs &a, const v4i (&acc)[FM][FN], const Tile &t, int row0,
                                         int lane, float *stg, const float *col_t, const float *col_b) {
    constexpr int BN = 16 * FN;
    static_assert(BN % 64 == 0, "staging needs whole 64-channel blocks");
    EpiCtx e;
    e.t = t;
    e.lane = lane;
    e.f32 = a.mode != 0;
    e.wh = e.f32 && a.form == 1;
    e.want_abs = e.f32 && a.next_absmax != nullptr && a.next_hblock > 0;
    e.inv_b = 1.0f / (float)a.hblock;
    e.ycols = e.f32 ? a.cout : a.cout_pad;
    e.ncols = e.ycols - t.n0 < BN ? e.ycols - t.n0 : BN;
    e.col_t = col_t;
    e.col_b = col_b;
    float wave_m = 0.0f;
    epilogue_groups<TW, FM, FN>(a, e, acc, row0, stg, wave_m, std::make_integer_sequence<int, FM>{});
    if (e.want_abs) {
        wave_m = wave_max(wave_m);
        if (lane == 0) atomic_max_nonneg(a.next_absmax + t.nb, wave_m);
    }
}

// Block index -> tile, XCD aware: blocks bid, bid+8, ... run on one XCD; each
// XCD gets a contiguous range of tiles so neighbouring tiles (which share input
// rows) share its L2.
__device__ __forceinline__ int xcd_logical_tile() {
    const int nt = gridDim.x;
    const int bid = blockIdx.x;
    const int xcd = bid & 7, q8 = nt >> 3, rmd = nt & 7;
    return xcd * q8 + (xcd < rmd ? xcd : rmd) + (bid >> 3);
}

// ---------------------------------------------------------------------------
// Small-cin path (cin_p <= 4, k*k*cin_p <= 128): K-steps of 64 contraction
// values gathered byte by byte (tap / channel from a lookup table), through
// registers into a double-buffered LDS tile.
// ---------------------------------------------------------------------------
template <int TH, int TW, int BN, int CIN_SMALL>
__global__ void __launch_bounds__(kThreads, 1) conv_gather_kernel(const ConvArgs a) {
    constexpr int BM = TH * TW;
    constexpr int TM = BM / 4;
    constexpr int FM = TM / 16;
    constexpr int FN = BN / 16;
    constexpr int A_PIECES = BM * 4 / kThreads;
    constexpr int B_PIECES = BN * 4 / kThreads;
    constexpr int BUF = (BM + BN) * 64;
    constexpr int EPI_BYTES = (4 * 16 + 2) * BN * 4;   // staging + column factors
    constexpr int LDS_BYTES = 2 * BUF > EPI_BYTES ? 2 * BUF : EPI_BYTES;
    static_assert(BM * 4 % kThreads == 0 && BN * 4 % kThreads == 0, "tile");
    __shared__ __attribute__((aligned(16))) int8_t lds[LDS_BYTES];
    __shared__ int s_lut_off[128];
    __shared__ int8_t s_lut_dh[128], s_lut_dw[128];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const Tile tile = block_tile(a, xcd_logical_tile(), TH, TW, BN);
    const int n0 = tile.n0;

    // per-thread A rows
    const int g = tid & 3;
    const int8_t *a_base[A_PIECES];
    int a_ih0[A_PIECES], a_iw0[A_PIECES];
#pragma unroll
    for (int p = 0; p < A_PIECES; ++p) {
        const int m = (tid >> 2) + 64 * p;
        const int gi = tile.gi0 + m / TW, gj = tile.gj0 + m % TW;
        if (gi < a.gh && gj < a.gw) {
            a_ih0[p] = gi * a.sa + a.bah;
            a_iw0[p] = gj * a.sa + a.baw;
            a_base[p] = a.xq + (int64_t)tile.nb * a.h * a.w * CIN_SMALL;
        } else {
            a_ih0[p] = -(1 << 28);   // every tap out of range
            a_iw0[p] = 0;
            a_base[p] = a.xq;
        }
    }

    // per contraction index d: tap offset and byte offset from the anchor pixel
    if (tid < 128) {
        const int d = tid;
        if (d < a.k_total) {
            const int t = d / CIN_SMALL, ci = d - t * CIN_SMALL;
            s_lut_dh[d] = a.dh[t];
            s_lut_dw[d] = a.dw[t];
            s_lut_off[d] = (a.dh[t] * a.w + a.dw[t]) * CIN_SMALL + ci;
        } else {
            // past the contraction: read the (bounds-checked) anchor pixel; the
            // prepared weights are zero there, so it contributes 0
            s_lut_dh[d] = 0;
            s_lut_dw[d] = 0;
            s_lut_off[d] = 0;
        }
    }
    __syncthreads();

    v4i ra[A_PIECES], rb[B_PIECES];
    auto global_load = [&](int ks) {
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
                acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fb[j], fa[i], acc[i][j], 0, 0, 0);
        if (ks + 1 < nks) lds_store(buf ^ 1);
        __syncthreads();
    }
    float *col = reinterpret_cast<float *>(lds) + 4 * 16 * BN;
    column_factors<BN>(a, tile, col, col + BN);
    __syncthreads();
    epilogue<TW, FM, FN>(a, acc, tile, wave * TM, lane, reinterpret_cast<float *>(lds) + wave * 16 * BN, col,
                         col + BN);
}

// Fill the tile counts of a launch over TH x TW tiles; returns the block count.
int64_t set_tiles(ConvArgs &b, int TH, int TW, int BN) {
    b.tiles_h = (b.gh + TH - 1) / TH;
    b.tiles_w = (b.gw + TW - 1) / TW;
    b.tiles_n = b.cout_pad / BN;
    return (int64_t)b.n * b.tiles_h * b.tiles_w * b.tiles_n;
}

template <int TH, int TW, int BN, int CS>
hipError_t launch_gather(const ConvArgs &a, hipStream_t st) {
    ConvArgs b = a;
    const int64_t tiles = set_tiles(b, TH, TW, BN);
    if (tiles <= 0 || tiles >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
    conv_gather_kernel<TH, TW, BN, CS><<<(unsigned)tiles, kThreads, 0, st>>>(b);
    return hipGetLastError();
}

template <int CS>
hipError_t launch_gather_n(const ConvArgs &a, hipStream_t st) {
    switch (a.cout_pad) {
        case 64: return launch_gather<8, 32, 64, CS>(a, st);
        case 128: return launch_gather<8, 32, 128, CS>(a, st);
        case 192: return launch_gather<8, 32, 192, CS>(a, st);
        case 256: return launch_gather<4, 32, 256, CS>(a, st);
        case 320: return launch_gather<4, 32, 320, CS>(a, st);
        default: return launch_gather<8, 32, 64, CS>(a, st);
    }
}

// ---------------------------------------------------------------------------
// Regular path (cin_p % 64 == 0): multi-stage pipeline.  A ring of STAGES LDS
// buffers, each holding one K-step's A tile (BM rows x 64 B) and B tile (BN x
// 64 B), is filled by buffer_load_dwordx4 ... lds (direct to LDS, no VGPRs).
// Each wave's DMA instruction writes 1 KB = 16 rows x 4 chunks contiguously;
// the lane that fills physical chunk p of row m fetches logical chunk
// p ^ swz(m).  Padding taps use an offset past the buffer's num_records, so the
// hardware returns zeros.  Per K-step: wait for this wave's DMAs of the next
// stage (vmcnt), one bare barrier (every wave's DMAs of that stage landed, and
// every wave is done with the buffer that gets refilled), issue the DMAs
// STAGES-1 steps ahead, then the MFMAs of this step while fragments of the
// next step stream into registers.
// ---------------------------------------------------------------------------
#define HATQ_LDS_PTR(p) ((__attribute__((address_space(3))) void *)(p))
constexpr uint32_t kOobOffset = 0x80000000u;   // beyond every buffer (< 2 GiB each)

__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, int8_t *lds_dst, uint32_t off) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, HATQ_LDS_PTR(lds_dst), 16, off, 0, 0, 0);
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt");
    // s_waitcnt simm16 (gfx9): vmcnt[3:0], expcnt[6:4]=7, lgkmcnt[11:8]=15, vmcnt_hi[15:14]
    __builtin_amdgcn_s_waitcnt((N & 15) | 0x70 | 0xF00 | ((N >> 4) << 14));
}

template <int TH, int TW, int BN, int STAGES>
__global__ void __launch_bounds__(kThreads, 1) conv_pipe_kernel(const ConvArgs a) {
    constexpr int BM = TH * TW;
    constexpr int TM = BM / 4;
    constexpr int FM = TM / 16;
    constexpr int FN = BN / 16;
    constexpr int A_INSTR = BM / 64;            // per wave per stage
    constexpr int B_INSTR = BN / 64;
    constexpr int PER_STAGE = A_INSTR + B_INSTR;
    constexpr int STAGE_BYTES = (BM + BN) * 64;
    static_assert(BM % 64 == 0 && BN % 64 == 0 && STAGES >= 3, "tile");
    static_assert(STAGES * STAGE_BYTES >= (4 * 16 + 2) * BN * 4, "epilogue staging fits in the ring");
    __shared__ __attribute__((aligned(1024))) int8_t lds[STAGES * STAGE_BYTES];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const Tile tile = block_tile(a, xcd_logical_tile(), TH, TW, BN);
    const int n0 = tile.n0;

    const int cin_p = a.cin_p;
    const int nchunks = cin_p >> 6;
    const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int8_t *>(a.xq), (short)0, (int)((int64_t)a.n * a.h * a.w * cin_p), 0x00020000);
    const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int8_t *>(a.wq), (short)0, (int)((int64_t)a.cout_pad * a.k_stride), 0x00020000);

    // A rows this lane fetches: instruction j covers rows 16*(wave + 4j) + lane/4
    int a_off[A_INSTR], a_ih0[A_INSTR], a_iw0[A_INSTR];
#pragma unroll
    for (int j = 0; j < A_INSTR; ++j) {
        const int m = 16 * (wave + 4 * j) + (lane >> 2);
        const int g = (lane & 3) ^ swz(m);
        const int gi = tile.gi0 + m / TW, gj = tile.gj0 + m % TW;
        if (gi < a.gh && gj < a.gw) {
            a_ih0[j] = gi * a.sa + a.bah;
            a_iw0[j] = gj * a.sa + a.baw;
            a_off[j] = ((tile.nb * a.h + a_ih0[j]) * a.w + a_iw0[j]) * cin_p + 16 * g;
        } else {
            a_ih0[j] = -(1 << 28);
            a_iw0[j] = 0;
            a_off[j] = 0;
        }
    }
    uint32_t b_off[B_INSTR];
#pragma unroll
    for (int j = 0; j < B_INSTR; ++j) {
        const int nn = 16 * (wave + 4 * j) + (lane >> 2);
        const int g = (lane & 3) ^ swz(nn);
        b_off[j] = (uint32_t)((n0 + nn) * a.k_stride + 16 * g);
    }

    auto issue = [&](int ks) {
        const int tap = ks / nchunks;
        const int chunk = ks - tap * nchunks;
        const int dh = a.dh[tap], dw = a.dw[tap];
        const int doff = (dh * a.w + dw) * cin_p + chunk * 64;
        int8_t *sb = lds + (ks % STAGES) * STAGE_BYTES;
#pragma unroll
        for (int j = 0; j < A_INSTR; ++j) {
            const int ih = a_ih0[j] + dh, iw = a_iw0[j] + dw;
            const bool in = (unsigned)ih < (unsigned)a.h && (unsigned)iw < (unsigned)a.w;
            dma16(rx, sb + 1024 * (wave + 4 * j), in ? (uint32_t)(a_off[j] + doff) : kOobOffset);
        }
        const uint32_t woff = (uint32_t)(a.wtap[tap] * cin_p + chunk * 64);
#pragma unroll
        for (int j = 0; j < B_INSTR; ++j) dma16(rw, sb + BM * 64 + 1024 * (wave + 4 * j), b_off[j] + woff);
    };

    v4i acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = v4i{0, 0, 0, 0};

    const int fr = lane & 15, fg = lane >> 4;
    // fragment addresses inside a stage buffer (loop invariant)
    int fa_off[FM], fb_off[FN];
#pragma unroll
    for (int i = 0; i < FM; ++i) {
        const int m = wave * TM + 16 * i + fr;
        fa_off[i] = m * 64 + 16 * (fg ^ swz(m));
    }
#pragma unroll
    for (int j = 0; j < FN; ++j) {
        const int nn = 16 * j + fr;
        fb_off[j] = BM * 64 + nn * 64 + 16 * (fg ^ swz(nn));
    }
    auto frag = [&](int ks, int off) {
        return *reinterpret_cast<const v4i *>(lds + (ks % STAGES) * STAGE_BYTES + off);
    };

    // B fragments stream through a ring of RING registers (RING-1 reads ahead,
    // continuing into stage ks+1); stage ks+1's A fragments go to the other A
    // set.  Reads that run past the last stage hit a stale in-bounds buffer and
    // are never used, so the MFMA block is unconditional.
    constexpr int RING = 4;
    static_assert(FN % RING == 0 && FN >= RING, "ring");
    const int nks = a.nksteps;
    v4i ring[RING];
    v4i fa0[FM], fa1[FM];

#pragma unroll
    for (int s = 0; s < STAGES - 1; ++s)
        if (s < nks) issue(s);
    if (STAGES - 2 < nks) wait_vmcnt<(STAGES - 2) * PER_STAGE>();
    else wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();
#pragma unroll
    for (int i = 0; i < FM; ++i) fa0[i] = frag(0, fa_off[i]);
#pragma unroll
    for (int r = 0; r < RING - 1; ++r) ring[r] = frag(0, fb_off[r]);

    auto stage = [&](int ks, v4i (&acur)[FM], v4i (&anext)[FM]) {
        if (ks + STAGES - 2 < nks) wait_vmcnt<(STAGES - 3) * PER_STAGE>();
        else wait_vmcnt<0>();
        __builtin_amdgcn_s_barrier();
        if (ks + STAGES - 1 < nks) issue(ks + STAGES - 1);
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const int jj = j + RING - 1;
            ring[jj % RING] = jj < FN ? frag(ks, fb_off[jj]) : frag(ks + 1, fb_off[jj - FN]);
            if (j >= FN - FM) anext[j - (FN - FM)] = frag(ks + 1, fa_off[j - (FN - FM)]);
#pragma unroll
            for (int i = 0; i < FM; ++i)
                acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(ring[j % RING], acur[i], acc[i][j], 0, 0, 0);
        }
    };
    // One stage per iteration (the A sets swap by copy): unrolling by two
    // stages makes the register allocator split the accumulators' live ranges.
    for (int ks = 0; ks < nks; ++ks) {
        stage(ks, fa0, fa1);
#pragma unroll
        for (int i = 0; i < FM; ++i) fa0[i] = fa1[i];
    }
    __syncthreads();   // every wave is done with the ring; reuse it as staging
    float *col = reinterpret_cast<float *>(lds) + 4 * 16 * BN;
    column_factors<BN>(a, tile, col, col + BN);
    __syncthreads();
    epilogue<TW, FM, FN>(a, acc, tile, wave * TM, lane, reinterpret_cast<float *>(lds) + wave * 16 * BN, col,
                         col + BN);
}

template <int TH, int TW, int BN, int STAGES>
hipError_t launch_pipe(const ConvArgs &a, hipStream_t st) {
    // keep every buffer under 2 GiB (32-bit buffer offsets, kOobOffset out of
    // range): launch over groups of whole samples
    const int64_t per_sample = (int64_t)a.h * a.w * a.cin_p;
    int64_t group = ((int64_t)1 << 31) / per_sample;
    if (group < 1) return hipErrorInvalidValue;
    if ((int64_t)a.cout_pad * a.k_stride >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
    for (int64_t s0 = 0; s0 < a.n; s0 += group) {
        ConvArgs b = a;
        const int gn = (int)(a.n - s0 < group ? a.n - s0 : group);
        b.n = gn;
        b.xq = a.xq + s0 * per_sample;
        b.sx = a.sx + s0;
        const int64_t out_per_sample = (int64_t)a.ho * a.wo * (a.mode == 0 ? a.cout_pad : a.cout);
        b.y = (void *)((char *)a.y + s0 * out_per_sample * 4);
        if (a.next_absmax) b.next_absmax = a.next_absmax + s0;
        b.M = (int64_t)gn * a.gh * a.gw;
        const int64_t tiles = set_tiles(b, TH, TW, BN);
        if (tiles <= 0 || tiles >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
        conv_pipe_kernel<TH, TW, BN, STAGES><<<(unsigned)tiles, kThreads, 0, st>>>(b);
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_conv(const ConvArgs &a, bool clear_next, hipStream_t st) {
    if (clear_next && a.next_absmax && a.next_hblock > 0)
        fill_u32_kernel<<<1, 256, 0, st>>>(reinterpret_cast<uint32_t *>(a.next_absmax), a.n, 0u);
    switch (a.cin_p <= 4 ? a.cin_p : 0) {
        case 0:
            switch (a.cout_pad) {
                case 64: return launch_pipe<8, 32, 64, 5>(a, st);
                case 128: return launch_pipe<8, 32, 128, 5>(a, st);
                case 192: return launch_pipe<8, 32, 192, 5>(a, st);
                case 256: return launch_pipe<4, 32, 256, 5>(a, st);
                case 320: return launch_pipe<4, 32, 320, 5>(a, st);
                default: return launch_pipe<8, 32, 64, 5>(a, st);
            }
        case 1: return launch_gather_n<1>(a, st);
        case 2: return launch_gather_n<2>(a, st);
        case 3: return launch_gather_n<3>(a, st);
        case 4: return launch_gather_n<4>(a, st);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace hatq
