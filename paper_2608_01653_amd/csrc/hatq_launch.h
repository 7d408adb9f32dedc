// Internal launchers of the HatQ kernels (host side, gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hatq {

// Activation transform + quantization of n samples of E floats each.
// absmax_in == nullptr: two passes through ws_absmax (n * kAbsSlots floats of
// scratch: the absmax pass's blocks of a sample spread their maxima over
// kAbsSlots slots, so no address takes more than a few atomics, and the
// quantization takes the maximum of the slots).
constexpr int kAbsSlots = 32;
// c64 > 0: the codes go out in the chunk-major layout of a sample of c64
// channels ([E / c64 pixels] per 64-channel plane; c64 % 64 == 0, hblock <= 64).
hipError_t launch_act_quant(const float *x, int n, int64_t E, int hblock, const float *absmax_in,
                            float *ws_absmax, int8_t *xq, float *act_scale, hipStream_t st, int c64 = 0);

// The same two-pass quantization with the per-sample absmax in the library's
// static device scratch (no caller workspace, no allocation): n <= kNoAllocMaxSamples
// (kNoAllocMaxSamples * kAbsSlots floats, 512 KB).
constexpr int kNoAllocMaxSamples = 4096;
hipError_t launch_act_quant_noalloc(const float *x, int n, int64_t E, int hblock, int8_t *xq, float *act_scale,
                                    hipStream_t st);

// Affine activation quantization (signed grid [-128, 127]) of n samples of E
// floats each (E % 4 == 0, the channel count a multiple of hblock): ws holds 2n
// floats (per-sample max(S, 0), then max(-S, 0)); per-sample scale and zero point out.
hipError_t launch_act_quant_affine(const float *x, int n, int64_t E, int hblock, float *ws, int8_t *xq,
                                   float *act_scale, int32_t *act_zero, hipStream_t st);

// Range-expansion profiling of n samples of P pixels x C channels: amax[k] =
// max |x|, amax[n + k] = max |S| (blocks of hblock, zero-padded), then the
// per-sample indicator into flags (or NULL) and its count added to *count (or
// NULL).  amax is 2n floats of caller memory.
hipError_t launch_range_expansion(const float *x, int n, int64_t P, int C, int hblock, float *amax, int32_t *flags,
                                  int32_t *count, hipStream_t st);

// Kronecker transform orders P_(m/16) (x) H~_16 the kernels implement, by the
// prime q of their Paley-I factor (order q + 1); 0 for other orders.
constexpr int kron_q(int m) { return m == 192 ? 11 : m == 320 ? 19 : 0; }

constexpr int kMaxTaps = 64;
constexpr int kModeIntTransition = 3;   // ConvArgs::mode of the integer transition

// Geometry and operands of one implicit-GEMM launch.  GEMM rows are the points
// (nb, gi, gj) of an n x gh x gw grid, processed in 2-D tiles of TH x TW points.  Input anchor of a point:
// (gi*sa + bah, gj*sa + baw); tap t reads the input pixel anchor + (dh[t], dw[t])
// with weight tap wtap[t] (kh*k + kw).  Output pixel: (gi*so + boh, gj*so + bow).
struct ConvArgs {
    const int8_t *xq;
    const int8_t *wp;      // K-blocked weights [pack_stride/64][cout_pad][64]
    const float *sx;
    const float *w_scale;
    const float *bias;
    void *y;               // NULL in F32 mode: only next_absmax is produced
    float *next_absmax;
    const float *q_absmax; // I8 mode: per-sample max |B_next y| giving the scale, or NULL
    float *q_scale;        // I8 mode: per-sample scale (written from q_absmax, else read)
    const int32_t *rq_table;   // mode 3: M [cout_pad], b_int [cout_pad], shift n
    const int32_t *zx;         // affine activations (modes 0, 1): per-sample zero point, or NULL
    const int32_t *tapsum;     // with zx: weight sums [k*k + 1][cout_pad] (per tap, then all taps)
    int64_t M;             // n * gh * gw
    int32_t n, h, w, cin_p;
    int32_t gh, gw;
    int32_t sa, bah, baw;
    int32_t ho, wo, so, boh, bow;
    int32_t k, ntaps, nksteps;   // kernel size; taps and K-steps of this launch
    int32_t k_total, pack_stride;
    int32_t rowrun;        // small-cin layer contracted per kernel row (16 B each)
    int32_t cout, cout_pad;
    int32_t form;          // 0 DH, 1 WH
    int32_t mode;          // 0 I32, 1 F32, 2 I8 (codes of B_next y, next_hblock the block),
                           // 3 the same codes by the integer transition (rq_table)
    int32_t hblock;        // the layer's block size
    int32_t next_hblock;   // 0 = no next-operand absmax
    int32_t paired;        // 1: a WH layer with next_hblock == hblock takes the next operand
                           // as z (B_next B_Cout = b I with identity nonlinearity); 0: both
                           // transforms run
    int32_t xq_c64;        // 1: xq in the chunk-major layout [n][cin_p/64][h][w][64]
    int32_t yq_c64;        // 1: code outputs in the chunk-major layout [n][cout/64][ho][wo][64]
    int32_t tiles_h, tiles_w, tiles_n;   // 2-D tiles of grid points per sample; column tiles
    int32_t n_base;        // first output column of a launch over a column range, else 0
    int32_t run_tiles;     // row-run kernel: tiles per block (set at launch)
    int8_t dh[kMaxTaps], dw[kMaxTaps];
    int16_t wtap[kMaxTaps];
};

// clear_next: zero next_absmax before the launch (false to keep accumulating
// across the phase launches of one transposed convolution).
hipError_t launch_conv(const ConvArgs &a, bool clear_next, hipStream_t st);

// Weight preparation: transform, per-channel scale, codes, bias.
struct PrepArgs {
    const float *w;        // PyTorch layout
    const float *bias;     // may be null
    int8_t *wq;
    float *w_scale;
    float *w_bias;
    int8_t *wpack;         // K-blocked copy of wq in the kernels' contraction order
    int32_t cin, cout, k, transposed, hblock, form;
    int32_t cin_p, cout_p, k_total, k_stride, pack_stride, rowrun;
};
hipError_t launch_prepare(const PrepArgs &a, hipStream_t st);
// Rebuild wpack from wq (geometry fields, wq and wpack are used).
hipError_t launch_pack(const PrepArgs &a, hipStream_t st);
// Per-tap weight sums of the codes: tapsum[t][c] = sum_ci wq[c][t*cin_p + ci] for
// t < k*k, and tapsum[k*k][c] = sum over all taps (geometry fields and wq used).
hipError_t launch_tapsums(const PrepArgs &a, int32_t *tapsum, hipStream_t st);

// Fixed-point parameters of the integer transition from static scales.
struct IntParamArgs {
    const float *w_scale;  // [cout_p]
    const float *bias;     // [cout_p], the prepared bias (WH: in the output basis)
    int32_t *table;        // out: M [cout_p], b_int [cout_p], shift n (-1: none fits)
    float s_x, s_y;
    int32_t cout_p;
    int32_t beta_in, beta_out;   // DH: (hblock, 1); WH: (1, hblock)
    int32_t K;                   // contraction length k*k*cin_p
    int32_t gain;                // WH output block times the next operand's block
};
hipError_t launch_int_params(const IntParamArgs &a, hipStream_t st);

}  // namespace hatq
