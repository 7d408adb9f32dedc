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
// Epilogue, in registers: a 64-channel block of one pixel lies in four lanes
// (see fwht_acc), so the dequantization (DH: y = fma(float(acc),
// fl(s_x*s_w,c)*(1/b), bias_c); WH: z/b = fma(float(acc), fl(s_x*s_w,c)*(1/b),
// b~_c/b); I32: raw), the WH output-basis restore (b-point FWHT) and the next
// layer's per-sample max |B_next y| run on the accumulators with no LDS round
// trip, and each lane stores 16 B of one pixel.
#include <utility>

#include "hatq_device.h"
#include "hatq_launch.h"

namespace hatq {
namespace {

constexpr int kThreads = 256;

// 16-B chunk swizzle of a 64-B LDS operand row (A and B tiles): chunk q of row
// f sits at position q ^ ((f >> 1) & 3).  A ds_read_b128 serves 8 lanes per
// pass from 32 banks; 8 consecutive rows then cover all 32 banks once, from any
// starting row, so fragment reads of consecutive rows are conflict-free.
__device__ __forceinline__ int swz(int row) { return (row >> 1) & 3; }

// A block's tile: sample nb, first grid point (gi0, gj0); local row m is the
// point (gi0 + m / TW, gj0 + m % TW).  Tiles never straddle samples.
struct Tile {
    int nb, gi0, gj0, n0;
};

__device__ __forceinline__ Tile block_tile(const ConvArgs &a, int logical, int TH, int TW, int BN) {
    Tile t;
    const int tile_m = logical / a.tiles_n;
    t.n0 = a.n_base + (logical - tile_m * a.tiles_n) * BN;
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

// Per-tile column factors of the dequantization (the tile is one sample, so
// s_x is uniform).  Both forms fold the factor 1/b in here:
//   DH: y = fma(acc, t_c, bias_c)        with t_c = fl(fl(s_x*s_w,c) / b) (b may be
//       a Kronecker order, 192 or 320; for a power of two this is exact scaling);
//   WH: z/b = fma(acc, t_c, b~_c * (1/b)), and y = B_Cout (z/b) = (B_Cout z)/b.
// Scaling by a power of two commutes with every rounding (results far above
// the subnormal range), so the WH output equals restoring z first and dividing
// after, as the operator is defined.
// In the integer transition (mode 3) the two slots carry the bits of the
// fixed-point multiplier M_c and of the integer bias b_int,c instead.
// The per-channel inputs of column c (scale and bias, or the integer
// transition's two table entries as bits) and the factors formed from them.
__device__ __forceinline__ void column_raw(const ConvArgs &a, int c, float &r0, float &r1) {
    if (a.mode == kModeIntTransition) {
        r0 = __int_as_float(a.rq_table[c]);
        r1 = __int_as_float(a.rq_table[a.cout_pad + c]);
    } else {
        r0 = a.w_scale[c];
        r1 = a.bias[c];
    }
}
__device__ __forceinline__ void column_from_raw(const ConvArgs &a, float sxv, float r0, float r1, float &t, float &b) {
    if (a.mode == kModeIntTransition) {
        t = r0;
        b = r1;
    } else if (a.form == 1) {
        const float inv_b = 1.0f / (float)a.hblock;
        t = (sxv * r0) * inv_b;
        b = r1 * inv_b;
    } else {
        t = (sxv * r0) / (float)a.hblock;   // exact scaling for a power of two
        b = r1;
    }
}
__device__ __forceinline__ void column_factor(const ConvArgs &a, float sxv, int c, float &t, float &b) {
    float r0, r1;
    column_raw(a, c, r0, r1);
    column_from_raw(a, sxv, r0, r1, t, b);
}

// The tile's activation scale (the integer transition has none).
__device__ __forceinline__ float tile_sx(const ConvArgs &a, int nb) {
    return a.mode == kModeIntTransition ? 0.0f : a.sx[nb];
}
// The same through the scalar unit (nb is wave-uniform): a scalar load is not
// counted by vmcnt, so it does not wait for the LDS DMAs and stores in flight.
__device__ __forceinline__ float tile_sx_uniform(const ConvArgs &a, int nb) {
    if (a.mode == kModeIntTransition) return 0.0f;
    const __attribute__((address_space(4))) float *p = (const __attribute__((address_space(4))) float *)a.sx;
    return p[__builtin_amdgcn_readfirstlane(nb)];
}

// Written by the whole block.
template <int BN>
__device__ __forceinline__ void column_factors(const ConvArgs &a, const Tile &t, float *col_t, float *col_b) {
    const float sxv = tile_sx(a, t.nb);
    for (int c = threadIdx.x; c < BN; c += kThreads) column_factor(a, sxv, t.n0 + c, col_t[c], col_b[c]);
}

// ---- register epilogue ------------------------------------------------------
// Channel c = n0 + 64*k + 16*jj + 4*q + r of the pixel of lane p + 16*q lies in
// acc[i][4*k + jj][r].  Inside a 64-channel block, channel bits 0-1 are the
// register r, bits 2-3 the lane bits 4-5 (q) and bits 4-5 the fragment jj: the
// quad layout of the activation kernels with the lane bits moved.  fwht_acc
// applies the same ascending-bit butterflies as fwht_item and produces the same
// fp32 values: every stage output is a correctly rounded a + c or a - c.

// Pair swap across lane bit 4 (MASK 16: odd 16-lane rows of x with even rows of
// y) or bit 5 (MASK 32: upper half of x with lower half of y).
template <int MASK>
__device__ __forceinline__ void pair_swap(float &x, float &y) {
    const unsigned xi = __float_as_uint(x), yi = __float_as_uint(y);
    if constexpr (MASK == 16) {
        const auto r = __builtin_amdgcn_permlane16_swap(xi, yi, false, false);
        x = __uint_as_float(r[0]);
        y = __uint_as_float(r[1]);
    } else {
        static_assert(MASK == 32, "lane bit 4 or 5");
        const auto r = __builtin_amdgcn_permlane32_swap(xi, yi, false, false);
        x = __uint_as_float(r[0]);
        y = __uint_as_float(r[1]);
    }
}

// Butterfly across lane bit MASK on all 16 registers, taken two at a time:
// after one pair swap every lane holds both partners (a: bit clear, c: bit
// set) of one pair, of the first register in the lanes with the bit clear and
// of the second in the others; a + c and a - c are formed in-lane.  With
// RESTORE a second swap puts them back in place; without it the values stay
// permuted among lanes and register pairs, which is enough where only their
// maximum is needed (the later stages pair registers r and r+4, r+8 and lanes
// l and l^32 in the same way in both layouts).
template <int MASK, bool RESTORE>
__device__ __forceinline__ void cross_stage_pairs(float (&v)[16]) {
#pragma unroll
    for (int r = 0; r < 16; r += 2) pair_swap<MASK>(v[r], v[r + 1]);
#pragma unroll
    for (int r = 0; r < 16; r += 2) {
        const float s = v[r] + v[r + 1], d = v[r] - v[r + 1];
        v[r] = s;
        v[r + 1] = d;
    }
    if constexpr (RESTORE) {
#pragma unroll
        for (int r = 0; r < 16; r += 2) pair_swap<MASK>(v[r], v[r + 1]);
    }
}

// Block size B <= 64 fixed at compile time (B = 1: no transform), so the
// stages are straight-line code.  All lanes of the wave must be active.
// B = -1: the block size b is taken at run time (wave-uniform branches); B = 0:
// no transform.
template <int B, bool RESTORE>
__device__ __forceinline__ void fwht_acc(float (&v)[16], int b) {
    static_assert(B == -1 || B == 0 || (B >= 1 && B <= 64 && (B & (B - 1)) == 0), "block size");
    if constexpr (B == -1) {
        if (b >= 2) reg_stage<1>(v);
        if (b >= 4) reg_stage<2>(v);
        if (b >= 8) cross_stage_pairs<16, RESTORE>(v);
        if (b >= 16) cross_stage_pairs<32, RESTORE>(v);
        if (b >= 32) reg_stage<4>(v);
        if (b >= 64) reg_stage<8>(v);
    } else {
        if constexpr (B >= 2) reg_stage<1>(v);
        if constexpr (B >= 4) reg_stage<2>(v);
        if constexpr (B >= 8) cross_stage_pairs<16, RESTORE>(v);
        if constexpr (B >= 16) cross_stage_pairs<32, RESTORE>(v);
        if constexpr (B >= 32) reg_stage<4>(v);
        if constexpr (B >= 64) reg_stage<8>(v);
    }
}

// max |B v| over the 16 values after fwht_acc<B, false>.  For B = 64 the last
// stage (registers r and r + 8) is fused with the maximum: of a + c and a - c,
// the one whose operands agree in sign has magnitude |a| + |c| and the other
// is no larger, and rounding is monotone, so max(|fl(a + c)|, |fl(a - c)|) =
// fl(|a| + |c|) exactly -- one add with absolute-value operands and one max
// per pair instead of an add, a subtract and two maxima.
template <int B>
__device__ __forceinline__ float fwht_acc_absmax(float (&v)[16], int b) {
    float mm = 0.0f;
    if constexpr (B == 64) {
        reg_stage<1>(v);
        reg_stage<2>(v);
        cross_stage_pairs<16, false>(v);
        cross_stage_pairs<32, false>(v);
        reg_stage<4>(v);
#pragma unroll
        for (int r = 0; r < 8; ++r) mm = fmaxf(mm, fabsf(v[r]) + fabsf(v[r + 8]));
    } else {
        fwht_acc<B, false>(v, b);
#pragma unroll
        for (int r = 0; r < 16; ++r) mm = fmaxf(mm, fabsf(v[r]));
    }
    return mm;
}

// ---- integer transition: the same butterflies on int64 values ---------------
// Integer butterflies are exact, so any stage order gives the Sylvester
// transform of the block; the layout and the lane pairing are those above.
template <int STRIDE>
__device__ __forceinline__ void reg_stage_i64(int64_t (&v)[16]) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        if (r & STRIDE) continue;
        const int64_t x = v[r], y = v[r + STRIDE];
        v[r] = x + y;
        v[r + STRIDE] = x - y;
    }
}

template <int MASK>
__device__ __forceinline__ void pair_swap_i64(int64_t &x, int64_t &y) {
    float xl = __uint_as_float((uint32_t)x), xh = __uint_as_float((uint32_t)((uint64_t)x >> 32));
    float yl = __uint_as_float((uint32_t)y), yh = __uint_as_float((uint32_t)((uint64_t)y >> 32));
    pair_swap<MASK>(xl, yl);
    pair_swap<MASK>(xh, yh);
    x = (int64_t)(((uint64_t)__float_as_uint(xh) << 32) | __float_as_uint(xl));
    y = (int64_t)(((uint64_t)__float_as_uint(yh) << 32) | __float_as_uint(yl));
}

template <int MASK>
__device__ __forceinline__ void cross_stage_i64(int64_t (&v)[16]) {
#pragma unroll
    for (int r = 0; r < 16; r += 2) pair_swap_i64<MASK>(v[r], v[r + 1]);
#pragma unroll
    for (int r = 0; r < 16; r += 2) {
        const int64_t x = v[r], y = v[r + 1];
        v[r] = x + y;
        v[r + 1] = x - y;
    }
#pragma unroll
    for (int r = 0; r < 16; r += 2) pair_swap_i64<MASK>(v[r], v[r + 1]);
}

// B as in fwht_acc (B = -1: block size b at run time; 0 or 1: none).
template <int B>
__device__ __forceinline__ void fwht_acc_i64(int64_t (&v)[16], int b) {
    const int bb = B == -1 ? b : B;
    if (bb >= 2) reg_stage_i64<1>(v);
    if (bb >= 4) reg_stage_i64<2>(v);
    if (bb >= 8) cross_stage_i64<16>(v);
    if (bb >= 16) cross_stage_i64<32>(v);
    if (bb >= 32) reg_stage_i64<4>(v);
    if (bb >= 64) reg_stage_i64<8>(v);
}

// clamp(rne(w / 2^n), -127, 127) for |w| < 2^62: adding 2^(n-1) - 1 plus the
// parity of the floor quotient rounds exact halves to the even neighbour.
__device__ __forceinline__ uint32_t int_code(int64_t w, int n, int64_t bias_m1) {
    const int64_t odd = n ? (w >> n) & 1 : 0;
    int64_t q = (w + bias_m1 + odd) >> n;
    q = q > 127 ? 127 : (q < -127 ? -127 : q);
    return (uint32_t)(int32_t)q;
}

// The same for n = 32 + s, s in [0, 30]: floor(w / 2^n) is the high word
// shifted right by s, so only the bias addition is 64-bit.
__device__ __forceinline__ uint32_t int_code_hi(int64_t w, int s, int64_t bias_m1) {
    const int32_t odd = ((int32_t)(w >> 32) >> s) & 1;
    const int64_t u = w + bias_m1 + odd;
    int32_t q = (int32_t)(u >> 32) >> s;
    q = q > 127 ? 127 : (q < -127 ? -127 : q);
    return (uint32_t)q;
}

// row0: the wave's first local row in the tile (local row m = row0 + 16*i + p is
// grid point (gi0 + m / TW, gj0 + m % TW)).  col_t / col_b: LDS column factors
// (column_factors, followed by a block barrier).
// Epilogue variants, fixed per kernel instantiation so that each kernel holds
// one straight-line body: WB is the block size of the WH restore (0: none) and
// NB the block size of the next operand's absmax (0: not wanted), both for
// fp32 output; WB = NB = -1 is the generic body, which takes the output mode,
// form and block sizes from the arguments.
// Q = 1: I8 output (the next operand's codes, NB its transform block); Q = 2:
// the same codes by the integer transition (mode 3); Q = 3: output from affine
// activation codes (fixed variants: F32 with no next-operand absmax, NB = 0;
// the generic one also I32); Q = 4: the next operand's absmax alone (F32 mode
// with no output).
template <int WB_, int NB_, int Q_ = 0>
struct Epi {
    static constexpr int WB = WB_, NB = NB_, Q = Q_;
};
using EpiGeneric = Epi<-1, -1>;
using EpiGenericInt = Epi<-1, -1, 2>;   // the integer transition, blocks at run time
using EpiGenericAffine = Epi<-1, -1, 3>;   // affine activations: zero-point correction
// A Kronecker order (192 or 320) for the WH restore or the next operand, on a
// tile of that many columns: float modes (Q = 5) and the integer transition
// (Q = 6).
using EpiKron = Epi<-1, -1, 5>;
using EpiKronInt = Epi<-1, -1, 6>;
using EpiKronAffine = Epi<-1, -1, 7>;   // the WH restore after the zero-point correction

// Orders the per-64-channel-block epilogue cannot apply, because the transform
// spans several of the lane's 64-channel blocks: the Kronecker orders and the
// Sylvester order 128.
inline bool wide_order(int b) { return kron_q(b) != 0 || b == 128; }

// Whether a launch applies such an order in its epilogue (any activation
// kind), and whether it takes the symmetric variants.
inline bool wide_needed(const ConvArgs &a) {
    const bool next = wide_order(a.next_hblock) &&
                      (a.next_absmax != nullptr || a.mode == 2 || a.mode == kModeIntTransition);
    const bool restore = a.form == 1 && wide_order(a.hblock) && a.mode != 0;
    return next || restore;
}
inline bool wide_epilogue(const ConvArgs &a) { return a.zx == nullptr && wide_needed(a); }

// The variant a launch needs, or the generic one.
template <typename E>
bool epi_matches(const ConvArgs &a) {
    if constexpr (E::WB == -1) {
        if constexpr (E::Q == 5 || E::Q == 6)
            return wide_epilogue(a) && (a.cout_pad == 192 || a.cout_pad == 320) &&
                   (a.mode == kModeIntTransition) == (E::Q == 6);
        if constexpr (E::Q == 7)
            return a.zx != nullptr && a.mode == 1 && wide_needed(a) && (a.cout_pad == 192 || a.cout_pad == 320);
        // (never a launch with a Kronecker order: a list without its variants
        // then finds no match and the launch fails)
        return (a.mode == kModeIntTransition) == (E::Q == 2) && (a.zx != nullptr) == (E::Q == 3) && !wide_needed(a);
    } else {
        if constexpr (E::Q == 5) {   // a Kronecker order at compile time (float modes)
            const int wb = a.form == 1 ? a.hblock : 0;
            const int nb = a.next_absmax != nullptr || a.mode == 2 ? a.next_hblock : 0;
            return wide_epilogue(a) && a.mode != kModeIntTransition && a.cout_pad % 64 == 0 && wb == E::WB &&
                   nb == E::NB;
        }
        if ((a.zx != nullptr) != (E::Q == 3)) return false;
        const int wb = a.form == 1 ? a.hblock : 0;
        if (E::Q == 3) return a.mode == 1 && wb == E::WB && a.next_absmax == nullptr;
        if (E::Q == 4)
            return a.mode == 1 && a.y == nullptr && a.next_absmax != nullptr && wb == E::WB && a.next_hblock == E::NB;
        if (E::Q == 1)   // the codes with the dynamic scale (from the next operand's absmax)
            return a.mode == 2 && a.q_absmax != nullptr && wb == E::WB && a.next_hblock == E::NB;
        if (E::Q) return a.mode == (E::Q == 2 ? kModeIntTransition : 2) && wb == E::WB && a.next_hblock == E::NB;
        const int nb = a.next_absmax != nullptr ? a.next_hblock : 0;
        return a.mode == 1 && wb == E::WB && nb == E::NB;
    }
}


template <typename E>
struct EpiFlags {
    static constexpr int WB = E::WB, NB = E::NB;
    static constexpr bool generic = WB == -1;
    // the Kronecker variants with fixed orders take the output mode at run time
    static constexpr bool flex = generic || E::Q == 5;
    bool f32, wh, want_abs, i8, iq, affine, store;
    __device__ explicit EpiFlags(const ConvArgs &a) {
        affine = E::Q == 3 || E::Q == 7;
        iq = E::Q == 2 || E::Q == 6;   // integer transition (its own variants, generic ones included)
        f32 = !iq && (generic ? a.mode != 0 : true);   // the fp32 arithmetic (F32 and I8 modes)
        wh = generic ? a.mode != 0 && a.form == 1 : WB != 0;
        want_abs = !iq && (flex ? a.mode == 1 && a.next_absmax != nullptr && a.next_hblock > 0
                                : (E::Q == 0 || E::Q == 4) && NB != 0);
        i8 = !iq && (flex ? a.mode == 2 : E::Q == 1);
        store = E::Q != 4 && !i8 && !iq && a.y != nullptr;   // I32 / F32 values
    }
};

// Stores 64-channel block k of group i: each lane writes 16 B (four channels)
// of its pixel per fragment.
template <int TW, int FN, typename E>
__device__ __forceinline__ void store_group_impl(const ConvArgs &a, const Tile &t, int row0, int lane, int i, int k,
                                                 const float (&v)[16]) {
    const int p = lane & 15, q = lane >> 4;
    const EpiFlags<E> fl(a);
    const int ycols = fl.f32 ? a.cout : a.cout_pad;
    const int ncols = ycols - t.n0 < 16 * FN ? ycols - t.n0 : 16 * FN;
    const int m = row0 + 16 * i + p;
    const int gi = t.gi0 + m / TW, gj = t.gj0 + m % TW;
    float *yp = reinterpret_cast<float *>(a.y) + out_pixel(a, t.nb, gi, gj) * ycols + t.n0;
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
        const int cl = 64 * k + 16 * jj + 4 * q;
        if ((ycols & 3) == 0) {
            // (plain stores: streaming ones made the layer-2 conv 5 % slower and
            // the next quantization 9 % faster, the step slower overall)
            if (cl < ncols)
                *reinterpret_cast<float4 *>(yp + cl) = make_float4(v[4 * jj], v[4 * jj + 1], v[4 * jj + 2], v[4 * jj + 3]);
        } else {
#pragma unroll
            for (int r = 0; r < 4; ++r)
                if (cl + r < ncols) yp[cl + r] = v[4 * jj + r];
        }
    }
}
#define store_group(a, t, row0, lane, i, k, v) store_group_impl<TW, FN, E>(a, t, row0, lane, i, k, v)

// Codes of 16 values as the activation quantizer rounds them: t = fl(u * r)
// rounded with the magic constant, and the IEEE quotient fl(u / s) for every
// value of a lane that has one near a half-integer (or when the scale is out of
// the fast path's range); w[jj] packs the codes of registers 4*jj .. 4*jj+3.
// (A per-register exact path behind a wave vote was measured slower: the
// branches split the straight-line code.)
// CLAMP = false when the scale comes from the values' own maximum (or an upper
// bound of it): then |u / s| <= 127 (1 + 2^-23) and every rounding stays in
// [-127, 127] without the clamp.
template <bool CLAMP = true>
__device__ __forceinline__ void quant16(const float (&u)[16], float s, float r, bool fast_ok, uint32_t (&w)[4]) {
    uint32_t c[16];
    bool near = !fast_ok;
#pragma unroll
    for (int k = 0; k < 16; ++k) {
        const float tq = CLAMP ? clamp127(u[k] * r) : u[k] * r;
        const float uf = tq + HATQ_MAGIC;
        const float kf = uf - HATQ_MAGIC;
        near |= fabsf(tq - kf) > HATQ_NEAR_TIE;
        c[k] = __float_as_uint(uf);
    }
    if (near) {
#pragma unroll
        for (int k = 0; k < 16; ++k) c[k] = __float_as_uint(rintf(clamp127(u[k] / s)) + HATQ_MAGIC);
    }
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) w[jj] = pack_low_bytes(c[4 * jj], c[4 * jj + 1], c[4 * jj + 2], c[4 * jj + 3]);
}

// The arithmetic: dequantization, WH restore, next-operand absmax (one atomic
// per wave at most) or, in I8 mode, the next operand's codes.  Each group is
// stored as soon as it is final (stores interleave with the arithmetic).  The
// work is split into the per-tile setup (constructor), one call per 64-channel
// block of the accumulators (block(acc, k), any order) and finish(), so a
// kernel can run a block's epilogue while later blocks' MFMAs are in flight.
template <int TW, int FM, int FN, typename E>
struct Epilogue {
    static_assert(FN % 4 == 0, "whole 64-channel blocks");
    static constexpr int WB = E::WB, NB = E::NB;
    static constexpr bool generic = WB == -1;
    static constexpr int NBLK = FN / 4;
    // the Kronecker order of a tile of 16 FN columns (192 = P_12 (x) H~_16,
    // 320 = P_20 (x) H~_16): its Paley q, and the values a lane holds per pixel
    static constexpr int KQ = FN == 12 ? 11 : FN == 20 ? 19 : 0;
    static constexpr int KB = 16 * FN, KV = 4 * FN;
    static constexpr bool kKron = (E::Q == 5 || E::Q == 6 || E::Q == 7) && KQ != 0;
    // The Sylvester order 128 on a tile of 128 or 256 columns (float modes,
    // orders at compile time): blocks of two 64-channel blocks of the lane.
    static constexpr bool kS128 = E::Q == 5 && E::WB != -1 && (E::WB == 128 || E::NB == 128);
    static_assert(!kS128 || (FN % 8 == 0 && !kKron), "order 128 on 128-column multiples");
    // the fixed I8 variants take the dynamic scale only (epi_matches): no clamp
    static constexpr bool kClamp = E::Q != 1;
    const ConvArgs &a;
    const Tile &t;
    const int row0, lane, p, q;
    const float *col_t, *col_b;
    const EpiFlags<E> fl;
    bool full, z_bound, zpair, q_fast, kron;
    float wave_m, seen, qs, qr;
    int nbk, rq_n, rq_pre, zp;
    int64_t rq_bias;
    uint64_t tapmask[FM];   // affine: the taps whose weight sums the pixel adjusts
    bool rq_pair, valid[FM], border[FM];

    __device__ __forceinline__ Epilogue(const ConvArgs &a_, const Tile &t_, int row0_, int lane_, const float *col_t_,
                                        const float *col_b_)
        : a(a_), t(t_), row0(row0_), lane(lane_), p(lane_ & 15), q(lane_ >> 4), col_t(col_t_), col_b(col_b_),
          fl(a_) {
        // the whole tile inside the grid (wave-uniform): no row masking needed
        full = t.gi0 + (row0 + 16 * FM - 1) / TW < a.gh && t.gj0 + TW <= a.gw;
        wave_m = 0.0f;
        // Published running maximum of this sample (read once; a stale value only
        // costs work).  A group whose rigorous upper bound on max |B_next y| stays
        // below it cannot raise the maximum, so its exact transform is skipped.
        seen = -1.0f;
        if (fl.want_abs) {
            if (lane == 0)
                seen = __uint_as_float(__hip_atomic_load(reinterpret_cast<unsigned int *>(a.next_absmax + t.nb),
                                                         __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
            seen = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(seen)));
        }
        nbk = generic ? a.next_hblock : NB;
        // WH layer whose next operand uses the same blocks, with the paired
        // cancellation allowed (identity between the layers): B y = B (B z / b)
        // = z exactly, so max|B y| <= max|z| (1 + 2 gamma_6 * 64) with gamma_6
        // the six-stage fp32 rounding factor (< 3.6e-7); 1 + 1e-4 covers it.
        // Without it every group runs both transforms.
        z_bound = a.paired && fl.wh && (generic ? a.hblock == a.next_hblock : WB == NB);
        // With no fp32 output to store, the next operand of such a layer is z
        // itself (B_next y = B B z / b = z in exact arithmetic): its maximum and
        // its codes are taken from z, and neither butterfly runs.
        zpair = !fl.affine && z_bound && !fl.store && nbk > 1 && (fl.want_abs || fl.i8);
        // A Kronecker order (192 = P_12 (x) H~_16, 320 = P_20 (x) H~_16) for the
        // next operand or the WH restore spans all the tile's 64-channel blocks
        // (a tile of that many columns: a lane holds every 16-channel group of
        // its pixel), so the Kronecker variants handle it after the last block
        // (block_kron).
        kron = false;
        if constexpr (kKron) {
            const bool nk = a.next_hblock == KB && (fl.want_abs || fl.i8 || fl.iq);
            kron = nk || (fl.wh && a.hblock == KB);
        }
        // I8 mode: the sample's scale (from the absmax as the activation quantizer
        // derives it, or given), published by the sample's first tile
        qs = 1.0f;
        qr = 1.0f;
        q_fast = true;
        if (fl.i8) {
            qs = a.q_absmax ? act_scale_from_absmax(a.q_absmax[t.nb]) : a.q_scale[t.nb];
            qr = 1.0f / qs;
            q_fast = qs >= 0x1p-125f && qs <= 0x1p125f;
            if (a.q_absmax && t.gi0 == 0 && t.gj0 == 0 && t.n0 == 0 && row0 == 0 && lane == 0) a.q_scale[t.nb] = qs;
        }
        // Integer transition: the shared shift n (in [0, 62]) after the two
        // tables.  A WH layer whose next operand uses the same blocks has
        // B_next B_Cout = b I on every kept block (Sylvester blocks square to b
        // times the identity; cout is a multiple of b, so truncation drops
        // whole blocks), so w = b p exactly: both transforms are skipped and
        // the shift absorbs log2(b) (a left shift rq_pre where n < log2(b)).
        rq_n = 0;
        rq_pre = 0;
        rq_bias = 0;
        rq_pair = false;
        if (fl.iq) {
            int n = __builtin_amdgcn_readfirstlane(a.rq_table[2 * a.cout_pad]);
            n = n < 0 ? 0 : (n > 62 ? 62 : n);   // the parameter call keeps n in [0, 62]
            rq_pair = a.paired && fl.wh && (generic ? a.hblock == a.next_hblock : WB == NB) && a.hblock > 1 &&
                      (a.hblock & (a.hblock - 1)) == 0;
            if (rq_pair) {
                const int lg = 31 - __builtin_clz(a.hblock);
                rq_pre = lg > n ? lg - n : 0;
                n = lg > n ? 0 : n - lg;
            }
            rq_n = n;
            rq_bias = n ? ((int64_t)1 << (n - 1)) - 1 : 0;
        }
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            const int m = row0 + 16 * i + p;
            valid[i] = t.gi0 + m / TW < a.gh && t.gj0 + m % TW < a.gw;
        }
        // Affine activations: the sample's zero point and, per row group, the
        // lane's taps to adjust (a launch with every tap: those outside the
        // image, subtracted from the total; a transposed phase: those inside,
        // added up), and whether any lane has one (wave-uniform).
        zp = 0;
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            border[i] = false;
            tapmask[i] = 0;
        }
        if (fl.affine) {
            zp = a.zx[t.nb];
            const bool all_taps = a.ntaps == a.k * a.k;
#pragma unroll
            for (int i = 0; i < FM; ++i) {
                const int m = row0 + 16 * i + p;
                const int ih0 = (t.gi0 + m / TW) * a.sa + a.bah, iw0 = (t.gj0 + m % TW) * a.sa + a.baw;
                uint64_t mk = 0;
                for (int tp = 0; tp < a.ntaps; ++tp) {
                    const int ih = ih0 + a.dh[tp], iw = iw0 + a.dw[tp];
                    const bool inside = ih >= 0 && ih < a.h && iw >= 0 && iw < a.w;
                    if (inside != all_taps) mk |= (uint64_t)1 << tp;
                }
                tapmask[i] = valid[i] ? mk : 0;
                border[i] = __builtin_amdgcn_ballot_w64(tapmask[i] != 0) != 0;
            }
        }
    }

    // Affine activations: codes outside the image read as 0, which stands for
    // the value -z s, so the centered sum is acc - z T(p, c), T the weight sum
    // over the launch's taps of pixel p that fall inside the image.  A launch
    // with every tap (regular convolution) starts from the total and removes
    // the outside taps of border pixels; a transposed phase adds its inside taps.
    __device__ __forceinline__ void zero_point_fix(v4i (&cc)[4], int i, int k) const {
        const int cl0 = t.n0 + 64 * k + 4 * q;
        const bool all_taps = a.ntaps == a.k * a.k;
        v4i T[4];
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) T[jj] = v4i{0, 0, 0, 0};
        if (all_taps) {
            const int32_t *full = a.tapsum + (int64_t)a.k * a.k * a.cout_pad + cl0;
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) T[jj] = *reinterpret_cast<const v4i *>(full + 16 * jj);
        }
        if (border[i]) {
            const int sg = all_taps ? -1 : 1;
            uint64_t mk = tapmask[i];
            while (mk) {
                const int tp = __builtin_ctzll(mk);
                mk &= mk - 1;
                const int wt = all_taps ? tp : a.wtap[tp];   // every tap: the table is the identity
                const int32_t *row = a.tapsum + (int64_t)wt * a.cout_pad + cl0;
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) T[jj] += sg * *reinterpret_cast<const v4i *>(row + 16 * jj);
            }
        }
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) cc[jj] -= zp * T[jj];
    }

    // Integer transition of block k: p = M (.) (acc + b_int) in int64, the WH
    // output transform, the next operand's transform, then the codes
    // clamp(rne(w / 2^n)).  Rows do not mix (the butterflies pair lanes of one
    // pixel), and channels past cout only meet channels past cout in the next
    // transform (cout is a multiple of its block), so neither needs masking.
    __device__ __forceinline__ void block_int(const v4i (&acc)[FM][FN], int k) {
        v4i m4[4], b4[4];
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
            const int cl = 64 * k + 16 * jj + 4 * q;
            m4[jj] = *reinterpret_cast<const v4i *>(col_t + cl);
            b4[jj] = *reinterpret_cast<const v4i *>(col_b + cl);
        }
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            int64_t v[16];
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
                const v4i c4 = acc[i][4 * k + jj];
#pragma unroll
                for (int r = 0; r < 4; ++r) v[4 * jj + r] = (int64_t)m4[jj][r] * (int64_t)(c4[r] + b4[jj][r]);
            }
            if (rq_pair) {
#pragma unroll
                for (int r = 0; r < 16; ++r) v[r] = (int64_t)((uint64_t)v[r] << rq_pre);
            } else {
                if (fl.wh) fwht_acc_i64<WB>(v, a.hblock);
                fwht_acc_i64<NB>(v, a.next_hblock);
            }
            // every lane forms its codes (the transpose in store_codes needs
            // them all); rows past the grid are not stored
            uint32_t c[16];
            if (rq_n >= 32) {
#pragma unroll
                for (int r = 0; r < 16; ++r) c[r] = int_code_hi(v[r], rq_n - 32, rq_bias);
            } else {
#pragma unroll
                for (int r = 0; r < 16; ++r) c[r] = int_code(v[r], rq_n, rq_bias);
            }
            uint32_t w[4];
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) w[jj] = pack_low_bytes(c[4 * jj], c[4 * jj + 1], c[4 * jj + 2], c[4 * jj + 3]);
            store_codes(w, i, k);
        }
    }

    // Codes of group (i, k): word jj of lane (p, q) holds channels 64k + 16jj + 4q
    // .. +3.  A 4 x 4 transpose of words between jj and the lane bits of q (pair
    // swaps across lane bits 5, then 4) gives lane (p, q) channels 64k + 16q ..
    // +15, stored as one 16-byte write.
    __device__ __forceinline__ void store_codes(uint32_t (&w)[4], int i, int k) const {
        auto swap32 = [](uint32_t &x, uint32_t &y) {
            const auto r = __builtin_amdgcn_permlane32_swap(x, y, false, false);
            x = r[0];
            y = r[1];
        };
        auto swap16 = [](uint32_t &x, uint32_t &y) {
            const auto r = __builtin_amdgcn_permlane16_swap(x, y, false, false);
            x = r[0];
            y = r[1];
        };
        swap32(w[0], w[2]);
        swap32(w[1], w[3]);
        swap16(w[0], w[1]);
        swap16(w[2], w[3]);
        if (!valid[i]) return;
        const int m = row0 + 16 * i + p;
        const int64_t pix = out_pixel(a, t.nb, t.gi0 + m / TW, t.gj0 + m % TW);
        int8_t *yq = reinterpret_cast<int8_t *>(a.y) + pix * a.cout + t.n0;
        if (a.yq_c64) {
            // chunk-major: block k of the tile is the plane (n0 + 64 k) / 64 of its sample
            const int64_t hw = (int64_t)a.ho * a.wo;
            yq = reinterpret_cast<int8_t *>(a.y) + ((int64_t)t.nb * (a.cout - 64) + t.n0 + 64 * k) * hw +
                 pix * 64 - 64 * k;
        }
        const int cl = 64 * k + 16 * q;
        // (the caller's buffer need only be 4-byte aligned: 16-byte writes when
        // every pixel's codes start 16-byte aligned, a launch-wide condition)
        const bool a16 = ((reinterpret_cast<uintptr_t>(a.y) | (uintptr_t)a.cout | (uintptr_t)t.n0) & 15) == 0;
        if (a16 && t.n0 + cl + 16 <= a.cout) {
            // streaming store: the next layer's convolution reads the codes
            __builtin_nontemporal_store(v4i{(int)w[0], (int)w[1], (int)w[2], (int)w[3]},
                                        reinterpret_cast<v4i *>(yq + cl));
        } else {
#pragma unroll
            for (int jj = 0; jj < 4; ++jj)
                if (t.n0 + cl + 4 * jj < a.cout) *reinterpret_cast<uint32_t *>(yq + cl + 4 * jj) = w[jj];
        }
    }

    // The sixteen values of 64-channel block k among a row group's KV.
    template <typename T>
    static __device__ __forceinline__ T (&grp(T (&v)[KV], int k))[16] {
        return *reinterpret_cast<T (*)[16]>(v + 16 * k);
    }

    // Float modes with a Kronecker order on the tile's KB columns.  Channel c
    // = 16 j + 4 q + r of the lane's pixel sits in v[4 j + r] (j = 4 k + jj the
    // fragment): the Kronecker index a * 16 + l has a = j (the Paley factor over
    // the FN fragments, in registers) and l = 4 q + r (the H~_16 factor:
    // register bits and lane bits 4-5, the first four stages of fwht_acc).  The
    // stage order is the activation kernel's (H~_16, then the Paley factor,
    // summed in ascending order), so the values are the ones it computes.
    __device__ void block_kron(const v4i (&acc)[FM][FN]) {
        const bool wh = fl.wh, want_abs = fl.want_abs, i8 = fl.i8, store = fl.store;
        // orders fixed at compile time (E::Q == 5 with WB, NB given): the WH
        // block 0 or the tile's order or a Sylvester block up to 64, the next
        // operand's 0, 1, the tile's order or a Sylvester block up to 64
        constexpr bool kFixed = E::WB != -1;
        constexpr int kWB = kFixed ? E::WB : 1, kNB = kFixed ? E::NB : 1;
        static_assert(!kFixed || ((kWB == 0 || kWB == KB || (kWB <= 64 && (kWB & (kWB - 1)) == 0)) &&
                                  (kNB <= 1 || kNB == KB || (kNB <= 64 && (kNB & (kNB - 1)) == 0))),
                      "fixed Kronecker variant orders");
        const int nb = kFixed ? kNB : a.next_hblock;
        // the lane's column-factor base (channel 4q of each 16), on the
        // 192-column tiles with a value the compiler cannot see through: with
        // its known low bits it turned base + offset into an or and kept one
        // address per channel group (spills in the window kernel; the 320-column
        // tile, with its accumulators in AGPRs, does better without)
        int qo = 4 * q;
        if constexpr (FN == 12) asm volatile("" : "+v"(qo));
        const float *ctq = col_t + qo, *cbq = col_b + qo;
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            float v[KV];
#pragma unroll
            for (int k = 0; k < NBLK; ++k) {
                v4i cc[4];
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) cc[jj] = acc[i][4 * k + jj];
                if (fl.affine) zero_point_fix(cc, i, k);
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) {
                    const int cl = 64 * k + 16 * jj;
                    const float4 t4 = *reinterpret_cast<const float4 *>(ctq + cl);
                    const float4 b4 = *reinterpret_cast<const float4 *>(cbq + cl);
                    v[16 * k + 4 * jj + 0] = __builtin_fmaf((float)cc[jj][0], t4.x, b4.x);
                    v[16 * k + 4 * jj + 1] = __builtin_fmaf((float)cc[jj][1], t4.y, b4.y);
                    v[16 * k + 4 * jj + 2] = __builtin_fmaf((float)cc[jj][2], t4.z, b4.z);
                    v[16 * k + 4 * jj + 3] = __builtin_fmaf((float)cc[jj][3], t4.w, b4.w);
                }
            }
            if (wh) {
                // the output restore: B^T z (the column factors carry 1/b)
                auto restore_kron = [&]() {
#pragma unroll
                    for (int k = 0; k < NBLK; ++k) fwht_acc<16, true>(grp(v, k), 16);
                    paley_stage_t<KQ>(v);
                };
                if constexpr (kFixed) {
                    if constexpr (kWB == KB) {
                        restore_kron();
                    } else if constexpr (kWB > 1) {
#pragma unroll
                        for (int k = 0; k < NBLK; ++k) fwht_acc<kWB, true>(grp(v, k), kWB);
                    }
                } else if (a.hblock == KB) {
                    restore_kron();
                } else {
#pragma unroll
                    for (int k = 0; k < NBLK; ++k) fwht_acc<-1, true>(grp(v, k), a.hblock);
                }
            }
            if (store && valid[i]) {
#pragma unroll
                for (int k = 0; k < NBLK; ++k) store_group(a, t, row0, lane, i, k, grp(v, k));
            }
            if (!(want_abs || i8)) continue;
            // rows past the grid are not part of the next operand (cout is a
            // multiple of the next block, so every channel is)
            if (!valid[i]) {
#pragma unroll
                for (int r = 0; r < KV; ++r) v[r] = 0.0f;
            }
            // channel order matters for the codes only
            auto next_kron = [&]() {
                if (i8) {
#pragma unroll
                    for (int k = 0; k < NBLK; ++k) fwht_acc<16, true>(grp(v, k), 16);
                } else {
#pragma unroll
                    for (int k = 0; k < NBLK; ++k) fwht_acc<16, false>(grp(v, k), 16);
                }
                paley_stage<KQ>(v);
            };
            if constexpr (kFixed) {
                if constexpr (kNB == KB) {
                    next_kron();
                } else if constexpr (kNB > 1) {
                    if (i8) {
#pragma unroll
                        for (int k = 0; k < NBLK; ++k) fwht_acc<kNB, true>(grp(v, k), kNB);
                    } else {
#pragma unroll
                        for (int k = 0; k < NBLK; ++k) fwht_acc<kNB, false>(grp(v, k), kNB);
                    }
                }
            } else if (nb == KB) {
                next_kron();
            } else if (nb > 1) {
                if (i8) {
#pragma unroll
                    for (int k = 0; k < NBLK; ++k) fwht_acc<-1, true>(grp(v, k), nb);
                } else {
#pragma unroll
                    for (int k = 0; k < NBLK; ++k) fwht_acc<-1, false>(grp(v, k), nb);
                }
            }
            if (i8) {
#pragma unroll
                for (int k = 0; k < NBLK; ++k) {
                    uint32_t w[4];
                    quant16(grp(v, k), qs, qr, q_fast, w);
                    store_codes(w, i, k);
                }
            } else {
                float mm = 0.0f;
#pragma unroll
                for (int r = 0; r < KV; ++r) mm = fmaxf(mm, fabsf(v[r]));
                wave_m = fmaxf(wave_m, mm);
            }
        }
    }

    // The integer transition with a Kronecker order (same layout; int64 is
    // exact, so the stage order is free).
    __device__ void block_int_kron(const v4i (&acc)[FM][FN]) {
        const int nb = a.next_hblock;
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            int64_t v[KV];
#pragma unroll
            for (int k = 0; k < NBLK; ++k)
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) {
                    const int cl = 64 * k + 16 * jj + 4 * q;
                    const v4i m4 = *reinterpret_cast<const v4i *>(col_t + cl);
                    const v4i b4 = *reinterpret_cast<const v4i *>(col_b + cl);
                    const v4i c4 = acc[i][4 * k + jj];
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        v[16 * k + 4 * jj + r] = (int64_t)m4[r] * (int64_t)(c4[r] + b4[r]);
                }
            if (fl.wh) {
                if (a.hblock == KB) {
#pragma unroll
                    for (int k = 0; k < NBLK; ++k) fwht_acc_i64<16>(grp(v, k), 16);
                    paley_stage_i64<KQ, true>(v);
                } else {
#pragma unroll
                    for (int k = 0; k < NBLK; ++k) fwht_acc_i64<-1>(grp(v, k), a.hblock);
                }
            }
            if (nb == KB) {
#pragma unroll
                for (int k = 0; k < NBLK; ++k) fwht_acc_i64<16>(grp(v, k), 16);
                paley_stage_i64<KQ, false>(v);
            } else {
#pragma unroll
                for (int k = 0; k < NBLK; ++k) fwht_acc_i64<-1>(grp(v, k), nb);
            }
#pragma unroll
            for (int k = 0; k < NBLK; ++k) {
                uint32_t c[16];
                if (rq_n >= 32) {
#pragma unroll
                    for (int r = 0; r < 16; ++r) c[r] = int_code_hi(v[16 * k + r], rq_n - 32, rq_bias);
                } else {
#pragma unroll
                    for (int r = 0; r < 16; ++r) c[r] = int_code(v[16 * k + r], rq_n, rq_bias);
                }
                uint32_t w[4];
#pragma unroll
                for (int jj = 0; jj < 4; ++jj)
                    w[jj] = pack_low_bytes(c[4 * jj], c[4 * jj + 1], c[4 * jj + 2], c[4 * jj + 3]);
                store_codes(w, i, k);
            }
        }
    }

    // 64-channel block k of every row group (one set of column factors serves all)
    __device__ __forceinline__ void block(const v4i (&acc)[FM][FN], int k) {
        if constexpr (kS128) {
            if (k == NBLK - 1) block_s128(acc);
        } else if constexpr (kKron && E::Q == 5 && E::WB != -1) {
            // orders fixed at compile time: always the Kronecker path
            if (k == NBLK - 1) block_kron(acc);
        } else {
            if constexpr (kKron) {
                if (kron) {
                    if (k == NBLK - 1) {
                        if (fl.iq) block_int_kron(acc);
                        else block_kron(acc);
                    }
                    return;
                }
            }
            block_plain(acc, k);
        }
    }

    // Float modes with the Sylvester order 128 for the WH restore and/or the next
    // operand (the other side a block up to 64 or none), after the tile's last
    // 64-channel block: the lane holds every 64-channel block of its pixel, so
    // a 128-block is the 64-point butterfly on blocks 2g and 2g + 1, then the
    // stage between them (channel bit 6, last: the activation kernel's
    // ascending stage order).
    __device__ void block_s128(const v4i (&acc)[FM][FN]) {
        constexpr int V = 4 * FN;
        const bool want_abs = fl.want_abs, i8 = fl.i8, store = fl.store;
        auto order128 = [](float (&v)[V], auto RESTOREc) {
            constexpr bool RESTORE = decltype(RESTOREc)::value;
#pragma unroll
            for (int k = 0; k < NBLK; ++k) fwht_acc<64, RESTORE>(grp(v, k), 64);
#pragma unroll
            for (int g = 0; g < V / 32; ++g)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const float x = v[32 * g + r], y = v[32 * g + 16 + r];
                    v[32 * g + r] = x + y;
                    v[32 * g + 16 + r] = x - y;
                }
        };
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            float v[V];
#pragma unroll
            for (int k = 0; k < NBLK; ++k)
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) {
                    const int cl = 64 * k + 16 * jj + 4 * q;
                    const float4 t4 = *reinterpret_cast<const float4 *>(col_t + cl);
                    const float4 b4 = *reinterpret_cast<const float4 *>(col_b + cl);
                    const v4i c4 = acc[i][4 * k + jj];
                    v[16 * k + 4 * jj + 0] = __builtin_fmaf((float)c4[0], t4.x, b4.x);
                    v[16 * k + 4 * jj + 1] = __builtin_fmaf((float)c4[1], t4.y, b4.y);
                    v[16 * k + 4 * jj + 2] = __builtin_fmaf((float)c4[2], t4.z, b4.z);
                    v[16 * k + 4 * jj + 3] = __builtin_fmaf((float)c4[3], t4.w, b4.w);
                }
            // the output restore B^T z = B z (the column factors carry 1/b)
            if constexpr (E::WB == 128) {
                order128(v, std::true_type{});
            } else if constexpr (E::WB > 1) {
#pragma unroll
                for (int k = 0; k < NBLK; ++k) fwht_acc<E::WB, true>(grp(v, k), E::WB);
            }
            if (store && valid[i]) {
#pragma unroll
                for (int k = 0; k < NBLK; ++k) store_group(a, t, row0, lane, i, k, grp(v, k));
            }
            if (!(want_abs || i8)) continue;
            // rows past the grid are not part of the next operand; channels
            // past cout neither
            const bool blk_full = t.n0 + 16 * FN <= a.cout;
            if (!valid[i] || !blk_full) {
#pragma unroll
                for (int k = 0; k < NBLK; ++k)
#pragma unroll
                    for (int jj = 0; jj < 4; ++jj)
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            const int ch = t.n0 + 64 * k + 16 * jj + 4 * q + r;
                            if (!valid[i] || ch >= a.cout) v[16 * k + 4 * jj + r] = 0.0f;
                        }
            }
            // channel order matters for the codes only
            if constexpr (E::NB == 128) {
                if (i8) order128(v, std::true_type{});
                else order128(v, std::false_type{});
            } else if constexpr (E::NB > 1) {
                if (i8) {
#pragma unroll
                    for (int k = 0; k < NBLK; ++k) fwht_acc<E::NB, true>(grp(v, k), E::NB);
                } else {
#pragma unroll
                    for (int k = 0; k < NBLK; ++k) fwht_acc<E::NB, false>(grp(v, k), E::NB);
                }
            }
            if (i8) {
#pragma unroll
                for (int k = 0; k < NBLK; ++k) {
                    uint32_t w[4];
                    quant16(grp(v, k), qs, qr, q_fast, w);
                    store_codes(w, i, k);
                }
            } else {
                float mm = 0.0f;
#pragma unroll
                for (int r = 0; r < V; ++r) mm = fmaxf(mm, fabsf(v[r]));
                wave_m = fmaxf(wave_m, mm);
            }
        }
    }

    // One 64-channel block of every row group, no Kronecker order.
    __device__ __forceinline__ void block_plain(const v4i (&acc)[FM][FN], int k) {
        if (fl.iq) {
            block_int(acc, k);
            return;
        }
        const bool f32 = fl.f32, wh = fl.wh, want_abs = fl.want_abs, i8 = fl.i8, store = fl.store;
        // The small-cin layer's two passes read the factors per group (LDS
        // reads are cheap next to its two transforms; kept across the row
        // groups they took 32 registers and the kernel spilled).
        constexpr bool serial = E::Q == 1 || E::Q == 4;
        float4 t4[4], b4[4];
        auto load_factors = [&]() {
            // zpair: the next operand is z itself, so the factors carry no 1/b
            // (t and b~ times b: exact, a power of two), and
            // fma(acc, t, b~) equals fma(acc, t/b, b~/b) * b
            const float bsc = zpair ? (float)a.hblock : 1.0f;
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
                const int cl = 64 * k + 16 * jj + 4 * q;
                t4[jj] = *reinterpret_cast<const float4 *>(col_t + cl);
                b4[jj] = *reinterpret_cast<const float4 *>(col_b + cl);
                if (zpair) {
                    t4[jj] = make_float4(t4[jj].x * bsc, t4[jj].y * bsc, t4[jj].z * bsc, t4[jj].w * bsc);
                    b4[jj] = make_float4(b4[jj].x * bsc, b4[jj].y * bsc, b4[jj].z * bsc, b4[jj].w * bsc);
                }
            }
        };
        if (f32 && !serial) load_factors();
        const bool blk_full = t.n0 + 64 * k + 64 <= a.cout;
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            // The requantizing and absmax-only variants (the small-cin layer's
            // two passes, with both transforms) keep one group's values live
            // at a time: interleaving groups spilled registers.
            if constexpr (serial) {
                __builtin_amdgcn_sched_barrier(0);
                if (f32) load_factors();
            }
            float v[16];
            v4i cc[4];
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) cc[jj] = acc[i][4 * k + jj];
            if (fl.affine) zero_point_fix(cc, i, k);
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
                const v4i c4 = cc[jj];
                if (!f32) {
#pragma unroll
                    for (int r = 0; r < 4; ++r) v[4 * jj + r] = __int_as_float(c4[r]);
                } else {
                    v[4 * jj + 0] = __builtin_fmaf((float)c4[0], t4[jj].x, b4[jj].x);
                    v[4 * jj + 1] = __builtin_fmaf((float)c4[1], t4[jj].y, b4[jj].y);
                    v[4 * jj + 2] = __builtin_fmaf((float)c4[2], t4[jj].z, b4[jj].z);
                    v[4 * jj + 3] = __builtin_fmaf((float)c4[3], t4[jj].w, b4[jj].w);
                }
            }
            if (zpair) {
                // v holds z
                if (i8) {
                    uint32_t w[4];
                    quant16<kClamp>(v, qs, qr, q_fast, w);
                    store_codes(w, i, k);
                } else {
                    // the maximum of |z| over the valid pixels and channels
                    // (wave-uniform branch: whole tiles take no masks)
                    float mm = 0.0f;
                    if (full && blk_full) {
#pragma unroll
                        for (int r = 0; r < 16; ++r) mm = fmaxf(mm, fabsf(v[r]));
                    } else {
#pragma unroll
                        for (int jj = 0; jj < 4; ++jj)
#pragma unroll
                            for (int r = 0; r < 4; ++r) {
                                const int ch = t.n0 + 64 * k + 16 * jj + 4 * q + r;
                                const bool in = valid[i] && ch < a.cout;
                                mm = fmaxf(mm, in ? fabsf(v[4 * jj + r]) : 0.0f);
                            }
                    }
                    wave_m = fmaxf(wave_m, mm);
                }
                continue;
            }
            // bound on this lane's share of max |B_next y| (see above)
            float zmax = 0.0f;
            if (want_abs && z_bound) {
#pragma unroll
                for (int r = 0; r < 16; ++r) zmax = fmaxf(zmax, fabsf(v[r]));
                zmax *= (float)a.hblock;   // v holds z / b
            }
            // (channels past cout are zeroed before the exact transform, which
            // breaks B y = z for a block that holds some)
            bool exact = want_abs;
            if (want_abs && nbk > 1 && z_bound && blk_full)
                exact = __builtin_amdgcn_ballot_w64(zmax * 1.0001f + 1e-30f >= seen) != 0;
            // the restored values are needed for a store, an exact maximum or codes
            if (wh && (store || exact || i8)) fwht_acc<WB, true>(v, a.hblock);   // the column factors carry the 1/b
            if (store && valid[i]) store_group(a, t, row0, lane, i, k, v);
            if (NB == 1 && exact) {
                // no transform: the maximum of |y| over the valid values
                const bool all = full && blk_full;
                float mm = 0.0f;
#pragma unroll
                for (int jj = 0; jj < 4; ++jj)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int ch = t.n0 + 64 * k + 16 * jj + 4 * q + r;
                        const bool in = all || (valid[i] && ch < a.cout);
                        mm = fmaxf(mm, in ? fabsf(v[4 * jj + r]) : 0.0f);
                    }
                wave_m = fmaxf(wave_m, mm);
            } else if (exact || i8) {
                // Rows past the grid and channels past cout are not part of the
                // next operand.
                if (!full || !blk_full) {
#pragma unroll
                    for (int jj = 0; jj < 4; ++jj)
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            const int ch = t.n0 + 64 * k + 16 * jj + 4 * q + r;
                            if (!valid[i] || ch >= a.cout) v[4 * jj + r] = 0.0f;
                        }
                }
                if (i8) {
                    // codes of B_next y in channel order (restoring butterflies)
                    fwht_acc<NB, true>(v, a.next_hblock);
                    uint32_t w[4];
                    quant16<kClamp>(v, qs, qr, q_fast, w);
                    store_codes(w, i, k);
                } else {
                    wave_m = fmaxf(wave_m, fwht_acc_absmax<NB>(v, a.next_hblock));
                }
            }
        }
    }

    __device__ __forceinline__ void finish() {
        if (fl.want_abs) {
            const float m = wave_max(wave_m);
            // The running maximum only grows, so a wave whose maximum does not exceed
            // a value already published skips its atomic.  Device-scope atomics on
            // one address serialize, and most waves of a layer end up skipping.
            if (lane == 0 && m > seen) atomic_max_nonneg(a.next_absmax + t.nb, m);
        }
    }
};

template <int TW, int FM, int FN, typename E>
__device__ __forceinline__ void epilogue_regs(const ConvArgs &a, const v4i (&acc)[FM][FN], const Tile &t,
                                              int row0, int lane, const float *col_t, const float *col_b) {
    Epilogue<TW, FM, FN, E> ep(a, t, row0, lane, col_t, col_b);
#pragma unroll
    for (int k = 0; k < FN / 4; ++k) ep.block(acc, k);
    ep.finish();
}

// Block index -> tile, XCD aware: blocks bid, bid+8, ... run on one XCD; each
// XCD gets a contiguous range of tiles so neighbouring tiles (which share input
// rows) share its L2.  xcd_tile maps a virtual block bid of a grid of nt.
__device__ __forceinline__ int xcd_tile(int bid, int nt) {
    const int xcd = bid & 7, q8 = nt >> 3, rmd = nt & 7;
    return xcd * q8 + (xcd < rmd ? xcd : rmd) + (bid >> 3);
}
__device__ __forceinline__ int xcd_logical_tile() { return xcd_tile(blockIdx.x, gridDim.x); }

// ---------------------------------------------------------------------------
// Row-run path (regular convolution, cin_p <= 4, k*cin_p <= 16, k <= 8,
// stride <= 2): in NHWC the taps kw = 0..k-1 of one kernel row kh are k*cin_p
// consecutive input bytes, so the contraction is taken as one 16-byte run per
// kernel row, d' = 16*kh + (kw*cin_p + ci) (weights zero past k*cin_p and past
// kh = k-1).  Lane group g of a fragment holds the run of kernel row 4*ks + g,
// read unaligned from an LDS copy of the input patch with byte funnel shifts.
//
// A block walks a run of RUN consecutive TH x TW tiles of one sample and one
// column tile: the weight tile and the column factors are staged once, and the
// next tile's patch is fetched while the current tile's epilogue runs (two
// patch buffers).  Accumulators stay small (two 16-point groups per wave) so
// two blocks share a CU.
// ---------------------------------------------------------------------------
// The input patch of a TH x TW tile of one sample nb in LDS: patch row r holds
// the input bytes of row ih0 + r from the 4-aligned address at or below its
// first byte (pixel iw0), fetched as aligned dwords; the row's alignment shift
// is (first byte address) mod 4.  load() issues every global load of a patch at
// once (no branches: rows outside the image use an out-of-range offset and
// read 0); store() applies the masks (bytes of columns inside both the patch
// and the image) and writes the LDS copy.  The range check drops the whole
// dword that straddles the end of the input; its bytes are read one by one.
template <int TH, int TW, int CIN>
struct RowRunPatch {
    static constexpr int PH = (TH - 1) * 2 + 8;                 // patch rows (stride <= 2, k <= 8)
    static constexpr int PWB = ((TW - 1) * 2 + 8) * CIN;        // patch bytes per row
    static constexpr int RS = (PWB + 3 + 20 + 15) / 16 * 16;    // LDS row stride: alignment shift + 20-byte reads
    static constexpr int RW = RS / 4;
    static constexpr int WORDS = PH * RW;
    static constexpr int PIT = (WORDS + kThreads - 1) / kThreads;

    const ConvArgs &a;
    const int nb;
    const int prow, pcols;   // patch rows and columns in use
    const int64_t in_bytes;
    const __amdgpu_buffer_rsrc_t rx;

    __device__ __forceinline__ RowRunPatch(const ConvArgs &a_, int nb_)
        : a(a_), nb(nb_), prow((TH - 1) * a_.sa + a_.k), pcols((TW - 1) * a_.sa + a_.k),
          in_bytes((int64_t)a_.n * a_.h * a_.w * CIN),
          rx(__builtin_amdgcn_make_buffer_rsrc(const_cast<int8_t *>(a_.xq), (short)0, (int)in_bytes, 0x00020000)) {}

    __device__ __forceinline__ int row_shift(int ih, int iw0) const {
        const uint32_t g = ((uint32_t)(nb * a.h + ih) * (uint32_t)a.w + (uint32_t)iw0) * (uint32_t)CIN;
        return (int)(g & 3u);
    }

    __device__ __forceinline__ void load(const Tile &tl, uint32_t (&pwd)[PIT]) const {
        const int tid = threadIdx.x;
        const int ih0 = tl.gi0 * a.sa + a.bah, iw0 = tl.gj0 * a.sa + a.baw;
#pragma unroll
        for (int it = 0; it < PIT; ++it) {
            const int e4 = tid + it * kThreads;
            const int r = e4 / RW, wi = e4 - r * RW;
            const int ih = ih0 + r;
            const bool live = e4 < WORDS && r < prow && (unsigned)ih < (unsigned)a.h;
            const int64_t ga = ((int64_t)(nb * a.h + ih) * a.w + iw0) * CIN + 4 * wi - row_shift(ih, iw0);
            pwd[it] = (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(rx, (int)(live ? (uint32_t)ga : 0xFFFFFFFFu),
                                                                     0, 0);
        }
    }

    __device__ __forceinline__ void store(const Tile &tl, const uint32_t (&pwd)[PIT], uint32_t *dst) const {
        const int tid = threadIdx.x;
        const int ih0 = tl.gi0 * a.sa + a.bah, iw0 = tl.gj0 * a.sa + a.baw;
        const int vlo = (iw0 < 0 ? -iw0 : 0) * CIN;
        const int vhi = (pcols < a.w - iw0 ? pcols : a.w - iw0) * CIN;
#pragma unroll
        for (int it = 0; it < PIT; ++it) {
            const int e4 = tid + it * kThreads;
            const int r = e4 / RW, wi = e4 - r * RW;
            const int ih = ih0 + r;
            const bool live = e4 < WORDS && r < prow && (unsigned)ih < (unsigned)a.h;
            const int rel0 = 4 * wi - row_shift(ih, iw0);   // byte index of byte 0 from pixel iw0
            const int64_t ga = ((int64_t)(nb * a.h + ih) * a.w + iw0) * CIN + rel0;
            uint32_t word = pwd[it];
            if (live && ga + 4 > in_bytes) {
                word = 0;
                for (int e = 0; e < 4 && ga + e < in_bytes; ++e)
                    word |= (uint32_t)(uint8_t)a.xq[ga + e] << (8 * e);
            }
            const int lo = live ? min(max(vlo - rel0, 0), 4) : 4, hi = min(max(vhi - rel0, 0), 4);
            const uint64_t keep = ((1ull << (8 * hi)) - 1) & ~((1ull << (8 * lo)) - 1);
            if (e4 < WORDS) dst[e4] = word & (uint32_t)keep;
        }
    }
};

// Tiles per block (a run of one sample): at least kRowRunMin; the launch
// raises it so the grid is about two blocks per CU (two fit a CU), one round
// with no tail, up to kRowRunMax.
constexpr int kRowRunMin = 4, kRowRunMax = 64;

template <int TH, int TW, int BN, int CIN, typename E, int MINB = 2>
__global__ void __launch_bounds__(kThreads, MINB) conv_rowrun_kernel(const ConvArgs a) {
    constexpr int BM = TH * TW;
    constexpr int TM = BM / 4;
    constexpr int FM = TM / 16;
    constexpr int FN = BN / 16;
    using P = RowRunPatch<TH, TW, CIN>;
    constexpr int RS = P::RS, PWORDS = P::WORDS, PIT = P::PIT;
    constexpr int BIT = 2 * BN * 4 / kThreads;
    static_assert(TM % 16 == 0 && TW % 16 == 0 && BN % 64 == 0 && 2 * BN * 4 % kThreads == 0, "tile");
    static_assert(BN <= kThreads, "one column per thread");
    __shared__ __attribute__((aligned(16))) int8_t s_b[2 * BN * 64];
    __shared__ uint32_t s_patch[2][PWORDS];
    __shared__ __attribute__((aligned(16))) float s_col[2 * BN];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int nks = a.nksteps;   // 1 or 2 (pack_stride / 64)

    // this block's run: sample nb, column tile n0, tiles t_first .. t_first+cnt-1
    // of the sample (row-major over tiles_h x tiles_w)
    const int per = a.tiles_h * a.tiles_w;
    const int run = a.run_tiles;
    const int runs = (per + run - 1) / run;
    const int logical = xcd_logical_tile();
    const int rn = logical / a.tiles_n;
    const int n0 = (logical - rn * a.tiles_n) * BN;
    const int nb = rn / runs;
    const int t_first = (rn - nb * runs) * run;
    const int cnt = per - t_first < run ? per - t_first : run;
    auto tile_of = [&](int t) {
        Tile tl;
        tl.nb = nb;
        tl.n0 = n0;
        const int th = t / a.tiles_w;
        tl.gi0 = th * TH;
        tl.gj0 = (t - th * a.tiles_w) * TW;
        return tl;
    };

    const P pp(a, nb);

    // ---- once per block: weight tile, column factors, first patch ----
    uint32_t pwd[PIT];
    {
        v4i wb[BIT];
#pragma unroll
        for (int it = 0; it < BIT; ++it) {
            const int pc = tid + it * kThreads;
            const int ks = pc / (BN * 4), rem = pc - ks * (BN * 4);
            wb[it] = v4i{0, 0, 0, 0};
            if (ks < nks)
                wb[it] = *reinterpret_cast<const v4i *>(a.wp + ((int64_t)ks * a.cout_pad + n0 + (rem >> 2)) * 64 +
                                                        16 * (rem & 3));
        }
        pp.load(tile_of(t_first), pwd);
        float colv_t = 0.0f, colv_b = 0.0f;
        if (tid < BN) column_factor(a, tile_sx(a, nb), n0 + tid, colv_t, colv_b);
#pragma unroll
        for (int it = 0; it < BIT; ++it) {
            const int pc = tid + it * kThreads;
            const int ks = pc / (BN * 4), rem = pc - ks * (BN * 4);
            const int nn = rem >> 2, g = rem & 3;
            *reinterpret_cast<v4i *>(s_b + ks * BN * 64 + nn * 64 + 16 * (g ^ swz(nn))) = wb[it];
        }
        if (tid < BN) {
            s_col[tid] = colv_t;
            s_col[BN + tid] = colv_b;
        }
        pp.store(tile_of(t_first), pwd, s_patch[0]);
    }
    __syncthreads();

    const int fr = lane & 15, fg = lane >> 4;
    for (int it = 0; it < cnt; ++it) {
        const Tile tile = tile_of(t_first + it);
        const bool more = it + 1 < cnt;
        if (more) pp.load(tile_of(t_first + it + 1), pwd);   // lands during this tile's work
        const uint32_t *patch = s_patch[it & 1];
        const int ih0 = tile.gi0 * a.sa + a.bah, iw0 = tile.gj0 * a.sa + a.baw;
        v4i acc[FM][FN];
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j) acc[i][j] = v4i{0, 0, 0, 0};
        for (int ks = 0; ks < nks; ++ks) {
            if (ks == 1 && a.k <= 6) {
                // Kernel rows 4 and 5 hold the only nonzero weights of this K-step:
                // a 32-deep MFMA (8 contraction bytes per lane, lane group fg ->
                // row 4 + fg/2, bytes 8*(fg&1) .. +7) does it at half the cost.
                const int kh = 4 + (fg >> 1), b0 = 8 * (fg & 1);
                long fa[FM];
#pragma unroll
                for (int i = 0; i < FM; ++i) {
                    const int m = wave * TM + 16 * i + fr;
                    const int ohl = m / TW, owl = m - ohl * TW;
                    const int row = a.sa * ohl + kh;
                    const int off = row * RS + a.sa * owl * CIN + b0 + pp.row_shift(ih0 + row, iw0);
                    const uint32_t *pw = patch + (off >> 2);
                    const uint32_t sh = off & 3;
                    const uint32_t d0 = pw[0], d1 = pw[1], d2 = pw[2];
                    const uint32_t lo = __builtin_amdgcn_alignbyte(d1, d0, sh), hi = __builtin_amdgcn_alignbyte(d2, d1, sh);
                    fa[i] = (long)(((uint64_t)hi << 32) | lo);
                }
#pragma unroll
                for (int j = 0; j < FN; ++j) {
                    const int nn = 16 * j + fr;
                    const long fb = *reinterpret_cast<const long *>(s_b + BN * 64 + nn * 64 + 16 * ((fg >> 1) ^ swz(nn)) + b0);
#pragma unroll
                    for (int i = 0; i < FM; ++i)
                        acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x32_i8(fb, fa[i], acc[i][j], 0, 0, 0);
                }
                continue;
            }
            // kernel row 4*ks + fg <= 7 stays inside the patch; rows >= k meet zero weights
            const int kh = 4 * ks + fg;
            v4i fa[FM];
#pragma unroll
            for (int i = 0; i < FM; ++i) {
                const int m = wave * TM + 16 * i + fr;
                const int ohl = m / TW, owl = m - ohl * TW;
                const int row = a.sa * ohl + kh;
                const int off = row * RS + a.sa * owl * CIN + pp.row_shift(ih0 + row, iw0);
                const uint32_t *pw = patch + (off >> 2);
                const uint32_t sh = off & 3;
                const uint32_t d0 = pw[0], d1 = pw[1], d2 = pw[2], d3 = pw[3], d4 = pw[4];
                fa[i] = v4i{(int)__builtin_amdgcn_alignbyte(d1, d0, sh), (int)__builtin_amdgcn_alignbyte(d2, d1, sh),
                            (int)__builtin_amdgcn_alignbyte(d3, d2, sh), (int)__builtin_amdgcn_alignbyte(d4, d3, sh)};
            }
#pragma unroll
            for (int j = 0; j < FN; ++j) {
                const int nn = 16 * j + fr;
                const v4i fb = *reinterpret_cast<const v4i *>(s_b + ks * BN * 64 + nn * 64 + 16 * (fg ^ swz(nn)));
#pragma unroll
                for (int i = 0; i < FM; ++i)
                    acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fb, fa[i], acc[i][j], 0, 0, 0);
            }
        }
        {
            // the epilogue reads the arguments and the lane afresh each tile
            // (through values the compiler cannot see through): hoisted out of
            // the tile loop they stay live through it and spill
            const __attribute__((address_space(4))) ConvArgs *kargs =
                (const __attribute__((address_space(4))) ConvArgs *)__builtin_amdgcn_kernarg_segment_ptr();
            asm volatile("" : "+s"(kargs));
            int elane = lane;
            asm volatile("" : "+v"(elane));
            epilogue_regs<TW, FM, FN, E>(*(const ConvArgs *)kargs, acc, tile, wave * TM, elane, s_col, s_col + BN);
        }
        // the other buffer was last read before the previous barrier
        if (more) pp.store(tile_of(t_first + it + 1), pwd, s_patch[(it + 1) & 1]);
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// The small-cin layer's two passes with both Table I transforms, on 32 x 32
// MFMA tiles: a WH layer with blocks of 64 whose output feeds a DH operand with
// blocks of 64, 192 output channels.  PASS 0 forms the next operand's
// per-sample max |B_next y| (no output); PASS 1 writes its codes with the scale
// derived from that maximum.  The contraction is the row-run one (one 16-byte
// run per kernel row) on v_mfma_i32_32x32x32_i8 with the weights as the first
// operand: lane (j, h), j = lane % 32 and h = lane / 32, supplies kernel row
// 2s + h of pixel j to MFMA s, and register r of 32-channel tile u holds
// channel 32u + 8(r/4) + 4h + r%4 of pixel j.
//
// A 64-channel block of one pixel is then 32 registers, index rho = 16u + r,
// of the lane pair (j, 0), (j, 1): channel bits 0, 1, 3, 4, 5 are bits 0-4 of
// rho and channel bit 2 is h, so each 64-point transform has five stages in
// registers and one across the lane halves (v_permlane32_swap).  That stage is
// left unrestored: pairing registers that differ in bit m, it leaves the stage's
// channel bit in register bit m and the lane half holding what bit m held.
// The WH restore pairs them by bit 1 (channel bit 1, already done), which
// leaves h = channel bit 1; the next transform's stage on channel bit 1 (now h)
// pairs them by bit 0, which leaves h = channel bit 0 and rho = channel bits
// 1-5: lane (j, h) ends with channels h + 2 rho of the block.  Both transforms
// keep the ascending stage order and the (a, c) -> (a + c, a - c) roundings of
// fwht_item, so the values are the ones the other kernels compute.
// ---------------------------------------------------------------------------
typedef int v16i __attribute__((ext_vector_type(16)));

// Butterfly across the lane halves on register pairs (rho, rho | M): after one
// swap the lanes with h = 0 hold both halves of register rho and those with
// h = 1 both halves of rho | M; a + c and a - c are formed in place.
template <int M>
__device__ __forceinline__ void half_stage(float (&v)[32]) {
#pragma unroll
    for (int r = 0; r < 32; ++r)
        if (!(r & M)) pair_swap<32>(v[r], v[r | M]);
#pragma unroll
    for (int r = 0; r < 32; ++r) {
        if (r & M) continue;
        const float s = v[r] + v[r | M], d = v[r] - v[r | M];
        v[r] = s;
        v[r | M] = d;
    }
}

// Codes rne(fl(v / s)) of N values whose scale comes from their own maximum, so
// |v / s| <= 127 (1 + 2^-23) and no clamp is needed.  Fast path: u = fl(v r +
// MAGIC) rounds the exact product v r to an integer k, and d = fl(v r - k)
// measures how far it lies from k.  With Q = v / s: |v r - Q| <= 127 * 2^-24
// (7.6e-6, r = fl(1/s)), |d - (v r - k)| <= 2^-25, and fl(Q) lies within half an
// ulp (<= 2^-18) of Q; so |d| <= 0.5 - 2^-16 puts fl(Q) strictly inside (k - 1/2,
// k + 1/2), and rne(fl(Q)) = k.  Values closer to a half-integer (or every value,
// for a scale outside the fast path's range) take the IEEE quotient, by groups
// of eight (one maximum of |d| per group), so a wave divides only the groups in
// which some lane needs it.  c[r] holds the code in its low byte.
template <int N>
__device__ __forceinline__ void rr32_codes(const float (&v)[N], float s, float r, bool fast_ok, uint32_t (&c)[N]) {
    static_assert(N % 8 == 0, "groups of eight");
    float dm[N / 8];
#pragma unroll
    for (int g = 0; g < N / 8; ++g) dm[g] = 0.0f;
#pragma unroll
    for (int i = 0; i < N; ++i) {
        const float uf = __builtin_fmaf(v[i], r, HATQ_MAGIC);
        const float kf = uf - HATQ_MAGIC;
        dm[i >> 3] = fmaxf(dm[i >> 3], fabsf(__builtin_fmaf(v[i], r, -kf)));
        c[i] = __float_as_uint(uf);
    }
    constexpr float kTie = 0.5f - 0x1p-16f;
#pragma unroll
    for (int g = 0; g < N / 8; ++g) {
        if (!fast_ok || dm[g] > kTie) {
#pragma unroll
            for (int i = 8 * g; i < 8 * g + 8; ++i) c[i] = __float_as_uint(rintf(clamp127(v[i] / s)) + HATQ_MAGIC);
        }
    }
}

// The codes of one 64-channel block of a grid point held by lane half h, from yq
// = the address of the block's first code + 16h: o[0..3] channels 16h .. +15,
// o[4..7] channels 32 + 16h .. +15, so each store instruction writes 32
// contiguous bytes per pixel (the two lanes of the pixel side by side).  16-byte
// stores where every pixel's codes start 16-byte aligned, else 4-byte ones.  NT:
// streaming stores (the next layer's convolution reads the codes, not this
// kernel).  The codes pass with both transforms measured 516 (streaming) against
// 532 us (plain); the paired pass, which issues its stores four times as
// densely, 623 against 307 us.
template <bool NT>
__device__ __forceinline__ void rr32_store(int8_t *yq, bool a16, const uint32_t (&o)[8]) {
    if (a16) {
        const v4i lo = v4i{(int)o[0], (int)o[1], (int)o[2], (int)o[3]}, hi = v4i{(int)o[4], (int)o[5], (int)o[6], (int)o[7]};
        if constexpr (NT) {
            __builtin_nontemporal_store(lo, reinterpret_cast<v4i *>(yq));
            __builtin_nontemporal_store(hi, reinterpret_cast<v4i *>(yq + 32));
        } else {
            *reinterpret_cast<v4i *>(yq) = lo;
            *reinterpret_cast<v4i *>(yq + 32) = hi;
        }
    } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            *reinterpret_cast<uint32_t *>(yq + 4 * q) = o[q];
            *reinterpret_cast<uint32_t *>(yq + 32 + 4 * q) = o[4 + q];
        }
    }
}

// Word exchange across the lane halves on the pairs (0, 2), (1, 3), (4, 6),
// (5, 7): the lanes with h = 0 then hold both halves' words 0, 1, 4, 5 (own in
// the first of each pair), those with h = 1 both halves' words 2, 3, 6, 7 (own
// in the second).
__device__ __forceinline__ void rr32_exchange(uint32_t (&w)[8]) {
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        if (q & 2) continue;
        const auto x = __builtin_amdgcn_permlane32_swap(w[q], w[q + 2], false, false);
        w[q] = x[0];
        w[q + 2] = x[1];
    }
}

// The same stages on int64 values (the integer transition): in registers, and
// across the lane halves with both 32-bit words swapped.
template <int STRIDE, int N>
__device__ __forceinline__ void reg_stage_i64n(int64_t (&v)[N]) {
#pragma unroll
    for (int r = 0; r < N; ++r) {
        if (r & STRIDE) continue;
        const int64_t x = v[r], y = v[r + STRIDE];
        v[r] = x + y;
        v[r + STRIDE] = x - y;
    }
}
template <int M>
__device__ __forceinline__ void half_stage_i64(int64_t (&v)[32]) {
#pragma unroll
    for (int r = 0; r < 32; ++r) {
        if (r & M) continue;
        uint32_t xl = (uint32_t)v[r], xh = (uint32_t)((uint64_t)v[r] >> 32);
        uint32_t yl = (uint32_t)v[r | M], yh = (uint32_t)((uint64_t)v[r | M] >> 32);
        const auto lo = __builtin_amdgcn_permlane32_swap(xl, yl, false, false);
        const auto hi = __builtin_amdgcn_permlane32_swap(xh, yh, false, false);
        const int64_t x = (int64_t)(((uint64_t)hi[0] << 32) | lo[0]);
        const int64_t y = (int64_t)(((uint64_t)hi[1] << 32) | lo[1]);
        v[r] = x + y;
        v[r | M] = x - y;
    }
}

// Output columns of a tile: one MFMA column set.
constexpr int kRr32W = 32;

// Codes of one 64-channel block of a pixel whose lane pair (j, 0), (j, 1)
// holds channel h + 2 rho in v[rho] (both transforms done), stored at yq: word
// w holds channels h + 8w + {0, 2, 4, 6}; after the exchange each pair (0, 2),
// (1, 3), (4, 6), (5, 7) holds the even and the odd channels of 8 consecutive
// ones, 16h + 8w' (+ 32 for the last two pairs), and a byte interleave puts them
// in order.
__device__ __forceinline__ void rr32_block_codes(const float (&v)[32], float qs, float qr, bool q_fast, bool valid,
                                                 int8_t *yq, bool a16) {
    uint32_t c[32];
    rr32_codes<32>(v, qs, qr, q_fast, c);
    uint32_t w[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) w[q] = pack_low_bytes(c[4 * q], c[4 * q + 1], c[4 * q + 2], c[4 * q + 3]);
    rr32_exchange(w);
    uint32_t o[8];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int e = q + (q & 2), d = e + 2;   // pairs (0, 2), (1, 3), (4, 6), (5, 7)
        o[2 * q] = __builtin_amdgcn_perm(w[d], w[e], 0x05010400u);       // [e0, o0, e1, o1]
        o[2 * q + 1] = __builtin_amdgcn_perm(w[d], w[e], 0x07030602u);   // [e2, o2, e3, o3]
    }
    if (valid) rr32_store<true>(yq, a16, o);
}

// half_stage<M> on each 32-value block of a lane's N values.
template <int M, int N>
__device__ __forceinline__ void half_stage_blocks(float (&v)[N]) {
    static_assert(N % 32 == 0, "32-value blocks");
#pragma unroll
    for (int r = 0; r < N; ++r)
        if (!(r & M)) pair_swap<32>(v[r], v[r | M]);
#pragma unroll
    for (int r = 0; r < N; ++r) {
        if (r & M) continue;
        const float s = v[r] + v[r | M], d = v[r] - v[r | M];
        v[r] = s;
        v[r | M] = d;
    }
}

// PAIRED (HATQ_PAIRED, the blocks equal): the next operand is z itself (B_next
// B_Cout = b I), so neither transform runs: the factors carry no 1/b (times b,
// exact), the maximum is max |z|, and the codes are those of z in the MFMA
// layout, where one swap of words across the lane halves gives each lane 32
// contiguous channels.
template <int TH, int CIN, int NS, int PASS, bool PAIRED, int MINB, int ORD = 64>
__global__ void __launch_bounds__(kThreads, MINB) conv_rr32_kernel(const ConvArgs a) {
    constexpr int TW = kRr32W, BN = 192, NBLK = BN / 64, RPW = TH / 4;
    // ORD: the order of both transforms (blocks of 64, or the order 192 on
    // all 192 channels: float passes only, both transforms explicit)
    static_assert(ORD == 64 || (ORD == 192 && PASS <= 1 && !PAIRED), "transform order");
    using P = RowRunPatch<TH, TW, CIN>;
    constexpr int RS = P::RS, PWORDS = P::WORDS, PIT = P::PIT;
    constexpr int WROWS = 2 * NS;   // kernel rows the MFMAs cover
    static_assert(TH % 4 == 0 && NS >= 1 && NS <= 4, "tile");
    __shared__ __attribute__((aligned(16))) int8_t s_w[WROWS * BN * 16];   // [kernel row][channel][16 B]
    __shared__ uint32_t s_patch[2][PWORDS];
    __shared__ __attribute__((aligned(16))) float s_col[2 * BN];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int j = lane & 31, h = lane >> 5;

    // this block's run: sample nb, tiles t_first .. t_first+cnt-1 of the sample
    const int per = a.tiles_h * a.tiles_w;
    const int run = a.run_tiles;
    const int runs = (per + run - 1) / run;
    const int rn = xcd_logical_tile();
    const int nb = rn / runs;
    const int t_first = (rn - nb * runs) * run;
    const int cnt = per - t_first < run ? per - t_first : run;
    auto tile_of = [&](int t) {
        Tile tl;
        tl.nb = nb;
        tl.n0 = 0;
        const int th = t / a.tiles_w;
        tl.gi0 = th * TH;
        tl.gj0 = (t - th * a.tiles_w) * TW;
        return tl;
    };
    const P pp(a, nb);

    // PASS 1: the sample's scale as the activation quantizer derives it,
    // published by the block whose run starts the sample
    // PASS 2: the shared shift n of the table (in [0, 62]); PAIRED: B_next B_Cout
    // = 64 I, so w = 64 p and the shift absorbs log2 64 (a left shift where n < 6)
    int rq_n = 0, rq_pre = 0;
    int64_t rq_bias = 0;
    if constexpr (PASS == 2) {
        int n = __builtin_amdgcn_readfirstlane(a.rq_table[2 * a.cout_pad]);
        n = n < 0 ? 0 : (n > 62 ? 62 : n);
        if constexpr (PAIRED) {
            rq_pre = 6 > n ? 6 - n : 0;
            n = 6 > n ? 0 : n - 6;
        }
        rq_n = n;
        rq_bias = n ? ((int64_t)1 << (n - 1)) - 1 : 0;
    }
    const float qs = PASS == 1 ? act_scale_from_absmax(a.q_absmax[nb]) : 1.0f;
    const float qr = 1.0f / qs;
    const bool q_fast = qs >= 0x1p-125f && qs <= 0x1p125f;
    if (PASS == 1 && t_first == 0 && tid == 0) a.q_scale[nb] = qs;

    // ---- once per block: weights, column factors, first patch ----
    uint32_t pwd[PIT];
    {
        // kernel row kh of channel c: 16 bytes of K-step kh / 4 of the packed weights
        constexpr int WIT = (WROWS * BN + kThreads - 1) / kThreads;
        v4i wb[WIT];
#pragma unroll
        for (int it = 0; it < WIT; ++it) {
            const int e = tid + it * kThreads;
            const int kh = e / BN, c = e - kh * BN;
            wb[it] = v4i{0, 0, 0, 0};
            if (e < WROWS * BN && kh < 4 * a.nksteps)
                wb[it] = *reinterpret_cast<const v4i *>(a.wp + ((int64_t)(kh >> 2) * a.cout_pad + c) * 64 +
                                                        16 * (kh & 3));
        }
        pp.load(tile_of(t_first), pwd);
        float colv_t = 0.0f, colv_b = 0.0f;
        if (tid < BN) column_factor(a, tile_sx(a, nb), tid, colv_t, colv_b);
        if constexpr (PAIRED && PASS != 2) {
            // z = fma(acc, t b, b~_c / b * b): the factors without the 1/b (b = 64)
            colv_t *= 64.0f;
            colv_b *= 64.0f;
        }
#pragma unroll
        for (int it = 0; it < WIT; ++it) {
            const int e = tid + it * kThreads;
            if (e < WROWS * BN) *reinterpret_cast<v4i *>(s_w + 16 * e) = wb[it];
        }
        if (tid < BN) {
            s_col[tid] = colv_t;
            s_col[BN + tid] = colv_b;
        }
        pp.store(tile_of(t_first), pwd, s_patch[0]);
    }
    __syncthreads();

    // 16-byte code stores when every pixel's codes start 16-byte aligned
    const bool a16 = PASS >= 1 && ((reinterpret_cast<uintptr_t>(a.y) | (uintptr_t)a.cout) & 15) == 0;
    float wave_m = 0.0f;
    for (int it = 0; it < cnt; ++it) {
        const Tile tile = tile_of(t_first + it);
        const bool more = it + 1 < cnt;
        if (more) pp.load(tile_of(t_first + it + 1), pwd);   // lands during this tile's work
        const uint32_t *patch = s_patch[it & 1];
        const int ih0 = tile.gi0 * a.sa + a.bah, iw0 = tile.gj0 * a.sa + a.baw;
#pragma unroll 1
        for (int rr = 0; rr < RPW; ++rr) {
            const int ohl = wave + 4 * rr;   // the wave's output row in the tile
            // pixel operand: kernel row 2s + h of pixel j, from the patch
            v4i fb[NS];
#pragma unroll
            for (int s = 0; s < NS; ++s) {
                const int row = a.sa * ohl + 2 * s + h;
                const int off = row * RS + a.sa * j * CIN + pp.row_shift(ih0 + row, iw0);
                const uint32_t *pw = patch + (off >> 2);
                const uint32_t sh = off & 3;
                const uint32_t d0 = pw[0], d1 = pw[1], d2 = pw[2], d3 = pw[3], d4 = pw[4];
                fb[s] = v4i{(int)__builtin_amdgcn_alignbyte(d1, d0, sh), (int)__builtin_amdgcn_alignbyte(d2, d1, sh),
                            (int)__builtin_amdgcn_alignbyte(d3, d2, sh), (int)__builtin_amdgcn_alignbyte(d4, d3, sh)};
            }
            const int gi = tile.gi0 + ohl, gj = tile.gj0 + j;
            const bool valid = gi < a.gh && gj < a.gw;
            // codes of block k at ybase + k * kstride (NHWC, or the chunk-major plane of block k)
            int8_t *ybase = nullptr;
            int64_t kstride = 64;
            if constexpr (PASS >= 1) {
                const int64_t pix = out_pixel(a, nb, gi, gj), hw = (int64_t)a.ho * a.wo;
                ybase = reinterpret_cast<int8_t *>(a.y) + 16 * h +
                        (a.yq_c64 ? (int64_t)nb * (a.cout - 64) * hw + pix * 64 : pix * a.cout);
                kstride = a.yq_c64 ? 64 * hw : 64;
            }
            if constexpr (ORD == 192) {
                // Order 192 = P_12 (x) H~_16 on both sides (the WH restore and
                // the next operand): all six 32-channel tiles of the pixel
                // first.  Register r of tile u holds channel c = 32u + 8
                // floor(r/4) + 4h + r mod 4: the H~_16 index l = c mod 16 has
                // bits 0-1 = r bits 0-1, bit 2 = h and bit 3 = r bit 2; the
                // Paley index a = c / 16 = 2u + r bit 3, so v[16u + r] is value
                // r mod 8 of group a at v[8a + r mod 8].  The stages are the
                // other kernels' (H~_16 in ascending bit order, then the Paley
                // factor summed in ascending order; transposed for the
                // restore), the lane-half stage left unrestored as for blocks of
                // 64, so each 64-channel block ends in the layout the codes
                // store takes (channel h + 2 rho).
                float v[96];
                // the weight fragments are the same for every row: an opaque
                // base keeps the compiler from holding all 18 (72 registers)
                // across the row loop
                int wbase = (h * BN + j) * 16;
                asm volatile("" : "+v"(wbase));
#pragma unroll
                for (int u = 0; u < 6; ++u) {
                    // one tile at a time: the dequantized values replace its
                    // accumulators
                    v16i acc = v16i{};
#pragma unroll
                    for (int s = 0; s < NS; ++s) {
                        const v4i fa = *reinterpret_cast<const v4i *>(s_w + wbase + (2 * s * BN + 32 * u) * 16);
                        acc = __builtin_amdgcn_mfma_i32_32x32x32_i8(fa, fb[s], acc, 0, 0, 0);
                    }
#pragma unroll
                    for (int q4 = 0; q4 < 4; ++q4) {
                        const int c0 = 32 * u + 8 * q4 + 4 * h;
                        const float4 t4 = *reinterpret_cast<const float4 *>(s_col + c0);
                        const float4 b4 = *reinterpret_cast<const float4 *>(s_col + BN + c0);
                        const int r0 = 16 * u + 4 * q4;
                        v[r0 + 0] = __builtin_fmaf((float)acc[4 * q4 + 0], t4.x, b4.x);
                        v[r0 + 1] = __builtin_fmaf((float)acc[4 * q4 + 1], t4.y, b4.y);
                        v[r0 + 2] = __builtin_fmaf((float)acc[4 * q4 + 2], t4.z, b4.z);
                        v[r0 + 3] = __builtin_fmaf((float)acc[4 * q4 + 3], t4.w, b4.w);
                    }
                }
                // the WH restore B^T (z / b) (the factors carry 1/b): H~_16,
                // then the transposed Paley factor
                reg_stage<1>(v);
                reg_stage<2>(v);
                half_stage_blocks<2>(v);   // l bit 2; then h = l bit 1
                reg_stage<4>(v);
                paley_stage_t<11>(v);
                // the next operand B_next y: H~_16 (l bit 1 now in h), then the
                // Paley factor
                reg_stage<1>(v);
                half_stage_blocks<1>(v);   // l bit 1; then h = l bit 0
                reg_stage<2>(v);
                reg_stage<4>(v);
                paley_stage<11>(v);
                if constexpr (PASS == 0) {
                    float mm = 0.0f;
#pragma unroll
                    for (int r = 0; r < 96; ++r) mm = fmaxf(mm, fabsf(v[r]));
                    wave_m = fmaxf(wave_m, valid ? mm : 0.0f);
                } else {
#pragma unroll
                    for (int k = 0; k < NBLK; ++k) {
                        float vk[32];
#pragma unroll
                        for (int r = 0; r < 32; ++r) vk[r] = v[32 * k + r];
                        rr32_block_codes(vk, qs, qr, q_fast, valid, ybase + k * kstride, a16);
                    }
                }
            } else {
#pragma unroll 1
            for (int k = 0; k < NBLK; ++k) {
                v16i acc[2];
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    acc[u] = v16i{};
#pragma unroll
                    for (int s = 0; s < NS; ++s) {
                        const v4i fa =
                            *reinterpret_cast<const v4i *>(s_w + ((2 * s + h) * BN + 64 * k + 32 * u + j) * 16);
                        acc[u] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fa, fb[s], acc[u], 0, 0, 0);
                    }
                }
                if constexpr (PASS == 2) {
                    // The integer transition (Table I, integer form): p = M_c (acc +
                    // b_int,c) in int64, the WH output transform, the next operand's
                    // transform, codes clamp(rne(w / 2^n)).  Integer butterflies are
                    // exact, so the stage order is free; the layout moves as in the
                    // float passes.  PAIRED: w = 64 p, no transform.
                    int64_t v[32];
#pragma unroll
                    for (int u = 0; u < 2; ++u)
#pragma unroll
                        for (int q4 = 0; q4 < 4; ++q4) {
                            const int c0 = 64 * k + 32 * u + 8 * q4 + 4 * h;
                            const v4i m4 = *reinterpret_cast<const v4i *>(s_col + c0);
                            const v4i b4 = *reinterpret_cast<const v4i *>(s_col + BN + c0);
#pragma unroll
                            for (int e = 0; e < 4; ++e)
                                v[16 * u + 4 * q4 + e] = (int64_t)m4[e] * (int64_t)(acc[u][4 * q4 + e] + b4[e]);
                        }
                    if constexpr (PAIRED) {
#pragma unroll
                        for (int r = 0; r < 32; ++r) v[r] = (int64_t)((uint64_t)v[r] << rq_pre);
                    } else {
                        reg_stage_i64n<1>(v);
                        reg_stage_i64n<2>(v);
                        half_stage_i64<2>(v);
                        reg_stage_i64n<4>(v);
                        reg_stage_i64n<8>(v);
                        reg_stage_i64n<16>(v);
                        reg_stage_i64n<1>(v);
                        half_stage_i64<1>(v);
                        reg_stage_i64n<2>(v);
                        reg_stage_i64n<4>(v);
                        reg_stage_i64n<8>(v);
                        reg_stage_i64n<16>(v);
                    }
                    uint32_t c[32];
                    if (rq_n >= 32) {
#pragma unroll
                        for (int r = 0; r < 32; ++r) c[r] = int_code_hi(v[r], rq_n - 32, rq_bias);
                    } else {
#pragma unroll
                        for (int r = 0; r < 32; ++r) c[r] = int_code(v[r], rq_n, rq_bias);
                    }
                    uint32_t w[8];
#pragma unroll
                    for (int q = 0; q < 8; ++q) w[q] = pack_low_bytes(c[4 * q], c[4 * q + 1], c[4 * q + 2], c[4 * q + 3]);
                    rr32_exchange(w);
                    if constexpr (PAIRED) {
                        if (valid)
                            rr32_store<false>(ybase + k * kstride, a16,
                                              {w[0], w[2], w[1], w[3], w[4], w[6], w[5], w[7]});
                    } else {
                        uint32_t o[8];
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            const int e = q + (q & 2), d = e + 2;
                            o[2 * q] = __builtin_amdgcn_perm(w[d], w[e], 0x05010400u);
                            o[2 * q + 1] = __builtin_amdgcn_perm(w[d], w[e], 0x07030602u);
                        }
                        if (valid) rr32_store<true>(ybase + k * kstride, a16, o);
                    }
                    continue;
                }
                if constexpr (PASS == 1 && PAIRED) {
                    // the codes of z, one 32-channel tile at a time (no stage
                    // mixes the tiles; all 32 values at once spilled)
                    uint32_t w[8];
#pragma unroll
                    for (int u = 0; u < 2; ++u) {
                        float z[16];
#pragma unroll
                        for (int q4 = 0; q4 < 4; ++q4) {
                            const int c0 = 64 * k + 32 * u + 8 * q4 + 4 * h;
                            const float4 t4 = *reinterpret_cast<const float4 *>(s_col + c0);
                            const float4 b4 = *reinterpret_cast<const float4 *>(s_col + BN + c0);
                            z[4 * q4 + 0] = __builtin_fmaf((float)acc[u][4 * q4 + 0], t4.x, b4.x);
                            z[4 * q4 + 1] = __builtin_fmaf((float)acc[u][4 * q4 + 1], t4.y, b4.y);
                            z[4 * q4 + 2] = __builtin_fmaf((float)acc[u][4 * q4 + 2], t4.z, b4.z);
                            z[4 * q4 + 3] = __builtin_fmaf((float)acc[u][4 * q4 + 3], t4.w, b4.w);
                        }
                        uint32_t c[16];
                        rr32_codes<16>(z, qs, qr, q_fast, c);
#pragma unroll
                        for (int q4 = 0; q4 < 4; ++q4)
                            w[4 * u + q4] = pack_low_bytes(c[4 * q4], c[4 * q4 + 1], c[4 * q4 + 2], c[4 * q4 + 3]);
                    }
                    // word 4u + q holds channels 32u + 8q + 4h .. +3; after the
                    // exchange the pairs (0, 2), (1, 3), (4, 6), (5, 7) hold the
                    // channels 32u + 16h + 8q' .. +7 in order
                    rr32_exchange(w);
                    if (valid)
                        rr32_store<false>(ybase + k * kstride, a16,
                                          {w[0], w[2], w[1], w[3], w[4], w[6], w[5], w[7]});
                    continue;
                }
                // dequantization (the factors carry 1/b), then the WH output
                // restore B^T (z / b)
                float v[32];
#pragma unroll
                for (int u = 0; u < 2; ++u)
#pragma unroll
                    for (int q4 = 0; q4 < 4; ++q4) {
                        const int c0 = 64 * k + 32 * u + 8 * q4 + 4 * h;
                        const float4 t4 = *reinterpret_cast<const float4 *>(s_col + c0);
                        const float4 b4 = *reinterpret_cast<const float4 *>(s_col + BN + c0);
                        const int r0 = 16 * u + 4 * q4;
                        v[r0 + 0] = __builtin_fmaf((float)acc[u][4 * q4 + 0], t4.x, b4.x);
                        v[r0 + 1] = __builtin_fmaf((float)acc[u][4 * q4 + 1], t4.y, b4.y);
                        v[r0 + 2] = __builtin_fmaf((float)acc[u][4 * q4 + 2], t4.z, b4.z);
                        v[r0 + 3] = __builtin_fmaf((float)acc[u][4 * q4 + 3], t4.w, b4.w);
                    }
                if constexpr (!PAIRED) {
                    reg_stage<1>(v);
                    reg_stage<2>(v);
                    half_stage<2>(v);
                    reg_stage<4>(v);
                    reg_stage<8>(v);
                    reg_stage<16>(v);
                    // the next operand: B_next y (pixels outside the grid are not
                    // part of it: their maximum is dropped and their codes not stored)
                    reg_stage<1>(v);
                    half_stage<1>(v);
                    reg_stage<2>(v);
                    reg_stage<4>(v);
                    reg_stage<8>(v);
                }
                if constexpr (PASS == 0 && PAIRED) {
                    float mm = 0.0f;
#pragma unroll
                    for (int r = 0; r < 32; ++r) mm = fmaxf(mm, fabsf(v[r]));
                    wave_m = fmaxf(wave_m, valid ? mm : 0.0f);
                } else if constexpr (PASS == 0) {
                    // last stage fused with the maximum: of a + c and a - c, the one
                    // whose operands agree in sign has magnitude |a| + |c| and the
                    // other is no larger; rounding is monotone, so
                    // max(|fl(a + c)|, |fl(a - c)|) = fl(|a| + |c|)
                    float mm = 0.0f;
#pragma unroll
                    for (int r = 0; r < 16; ++r) mm = fmaxf(mm, fabsf(v[r]) + fabsf(v[r + 16]));
                    wave_m = fmaxf(wave_m, valid ? mm : 0.0f);
                } else {
                    if constexpr (!PAIRED) reg_stage<16>(v);
                    rr32_block_codes(v, qs, qr, q_fast, valid, ybase + k * kstride, a16);
                }
            }
            }
        }
        // the other buffer was last read before the previous barrier
        if (more) pp.store(tile_of(t_first + it + 1), pwd, s_patch[(it + 1) & 1]);
        __syncthreads();
    }
    if constexpr (PASS == 0) {
        // one atomic per wave and run (a run is one sample); the running maximum
        // only grows, so a wave that does not exceed the published value skips it
        const float m = wave_max(wave_m);
        if (lane == 0 && m > __uint_as_float(__hip_atomic_load(reinterpret_cast<unsigned int *>(a.next_absmax + nb),
                                                                __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)))
            atomic_max_nonneg(a.next_absmax + nb, m);
    }
}

// ---------------------------------------------------------------------------
// Small-cin path (cin_p <= 4, k*k*cin_p <= 128): K-steps of 64 contraction
// values gathered byte by byte (tap / channel from a lookup table), through
// registers into a double-buffered LDS tile.
// ---------------------------------------------------------------------------
template <int TH, int TW, int BN, int CIN_SMALL, typename E>
__global__ void __launch_bounds__(kThreads, 1) conv_gather_kernel(const ConvArgs a) {
    constexpr int BM = TH * TW;
    constexpr int TM = BM / 4;
    constexpr int FM = TM / 16;
    constexpr int FN = BN / 16;
    constexpr int A_PIECES = BM * 4 / kThreads;
    constexpr int B_PIECES = BN * 4 / kThreads;
    constexpr int BUF = (BM + BN) * 64;
    constexpr int LDS_BYTES = 2 * BUF;
    static_assert(LDS_BYTES >= 2 * BN * 4, "column factors fit");
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
            rb[p] = *reinterpret_cast<const v4i *>(a.wp + ((int64_t)ks * a.cout_pad + n0 + nn) * 64 + g * 16);
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
    float *col = reinterpret_cast<float *>(lds);
    column_factors<BN>(a, tile, col, col + BN);
    __syncthreads();
    epilogue_regs<TW, FM, FN, E>(a, acc, tile, wave * TM, lane, col, col + BN);
}

// Fill the tile counts of a launch over TH x TW tiles; returns the block count.
int64_t set_tiles(ConvArgs &b, int TH, int TW, int BN) {
    b.tiles_h = (b.gh + TH - 1) / TH;
    b.tiles_w = (b.gw + TW - 1) / TW;
    b.tiles_n = b.cout_pad / BN;
    return (int64_t)b.n * b.tiles_h * b.tiles_w * b.tiles_n;
}

// Launch with the first epilogue variant of Es that matches (the last must be
// EpiGeneric, taken for anything the others do not match).
template <typename E, typename... Es, typename L>
hipError_t with_epilogue(const ConvArgs &a, L &&launch) {
    if constexpr (sizeof...(Es) == 0) {
        static_assert(E::WB == -1 && E::Q == 0, "the generic variant comes last");
        if (!epi_matches<E>(a)) return hipErrorInvalidValue;   // a Kronecker order this list lacks
        return launch(E{});
    } else {
        if (epi_matches<E>(a)) return launch(E{});
        return with_epilogue<Es...>(a, launch);
    }
}

// Variants compiled for the layer shapes of the analysis transforms: DH or WH
// blocks of 64, next operand blocked by 64 (DH next), 1 (WH next) or none.
#define HATQ_GENERIC_EPILOGUES EpiGenericInt, EpiGenericAffine, EpiGeneric
#define HATQ_KRON_EPILOGUES EpiKron, EpiKronInt, EpiKronAffine
// The float-mode Kronecker variants with the orders at compile time, per tile
// width (the paper's orders on every layer of a stack: order 192 on both sides
// of a 192-column layer, 320 on a 320-column one).
#define HATQ_KRON192_FIXED Epi<0, 192, 5>, Epi<192, 192, 5>, Epi<192, 1, 5>, Epi<192, 0, 5>
#define HATQ_KRON320_FIXED Epi<0, 320, 5>, Epi<320, 1, 5>, Epi<320, 0, 5>
// The Sylvester order 128 (tiles of 128 or 256 columns).
#define HATQ_S128_FIXED \
    Epi<128, 0, 5>, Epi<128, 1, 5>, Epi<128, 128, 5>, Epi<0, 128, 5>, Epi<64, 128, 5>, Epi<128, 64, 5>

int persistent_blocks();

template <int TH, int TW, int BN, int CS, typename E, int MINB = 2>
hipError_t launch_rowrun(const ConvArgs &a, hipStream_t st) {
    ConvArgs b = a;
    const int64_t tiles = set_tiles(b, TH, TW, BN);
    if (tiles <= 0 || b.nksteps < 1 || b.nksteps > 2 || b.sa > 2 || b.k > 8) return hipErrorInvalidValue;
    // every byte offset of the input fits the 32-bit buffer range
    if ((int64_t)b.n * b.h * b.w * CS >= ((int64_t)1 << 31) - 64) return hipErrorInvalidValue;
    const int64_t per = (int64_t)b.tiles_h * b.tiles_w;
    const int64_t slots = MINB * (int64_t)persistent_blocks();   // resident blocks (0 if unknown)
    int64_t run = slots > 0 ? (b.n * per * b.tiles_n + slots - 1) / slots : kRowRunMin;
    run = run < kRowRunMin ? kRowRunMin : run > kRowRunMax ? kRowRunMax : run;
    b.run_tiles = (int32_t)run;
    const int64_t blocks = (int64_t)b.n * ((per + run - 1) / run) * b.tiles_n;
    if (blocks >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
    conv_rowrun_kernel<TH, TW, BN, CS, E, MINB><<<(unsigned)blocks, kThreads, 0, st>>>(b);
    return hipGetLastError();
}

// The launch conv_rr32_kernel implements: 0 (absmax pass), 1 (codes), or -1.
// Three input channels, 192 output channels, 5x5 or 6x6 kernels (kernel rows
// 0-5 on three MFMAs), a WH layer with blocks of 64 into a next operand with
// blocks of 64 (both transforms, or with HATQ_PAIRED neither).
inline int rr32_pass(const ConvArgs &a) {
    if (!a.rowrun || a.cin_p != 3 || a.cout != 192 || a.cout_pad != 192 || a.n_base != 0) return -1;
    if (a.k < 5 || a.k > 6 || a.sa > 2 || a.nksteps != 2) return -1;
    if (a.form != 1 || a.hblock != 64 || a.next_hblock != 64 || a.zx != nullptr) return -1;
    if (a.mode == 1 && a.y == nullptr && a.next_absmax != nullptr) return 0;
    if (a.mode == 2 && a.q_absmax != nullptr) return 1;
    if (a.mode == kModeIntTransition) return 2;
    return -1;
}

// The same with the order 192 = P_12 (x) H~_16 (m(192), the paper's order for
// 192 channels) on both sides instead of blocks of 64: 0, 1, or -1.
inline int rr32_kron_pass(const ConvArgs &a) {
    if (!a.rowrun || a.cin_p != 3 || a.cout != 192 || a.cout_pad != 192 || a.n_base != 0) return -1;
    if (a.k < 5 || a.k > 6 || a.sa > 2 || a.nksteps != 2) return -1;
    if (a.form != 1 || a.hblock != 192 || a.next_hblock != 192 || a.zx != nullptr || a.paired) return -1;
    if (a.mode == 1 && a.y == nullptr && a.next_absmax != nullptr) return 0;
    if (a.mode == 2 && a.q_absmax != nullptr) return 1;
    return -1;
}

#ifndef HATQ_RR32_TH
#define HATQ_RR32_TH 16
#endif
#ifndef HATQ_RR32_MINB
#define HATQ_RR32_MINB 4
#endif
// the integer transition (int64 values: twice the registers; 159 VGPRs, three
// blocks per CU)
#ifndef HATQ_RR32_MINB_INT
#define HATQ_RR32_MINB_INT 3
#endif
// the order 192 (a pixel's 96 values per lane at once)
#ifndef HATQ_RR32_MINB_KRON
#define HATQ_RR32_MINB_KRON 2
#endif

template <int TH, int NS, int PASS, bool PAIRED, int MINB, int ORD = 64>
hipError_t launch_rr32(const ConvArgs &a, hipStream_t st) {
    ConvArgs b = a;
    const int64_t tiles = set_tiles(b, TH, kRr32W, 192);
    if (tiles <= 0 || (ORD == 64 ? rr32_pass(b) : rr32_kron_pass(b)) != PASS || (b.paired != 0) != PAIRED)
        return hipErrorInvalidValue;
    // every byte offset of the input fits the 32-bit buffer range
    if ((int64_t)b.n * b.h * b.w * 3 >= ((int64_t)1 << 31) - 64) return hipErrorInvalidValue;
    const int64_t per = (int64_t)b.tiles_h * b.tiles_w;
    const int64_t slots = MINB * (int64_t)persistent_blocks();   // resident blocks (0 if unknown)
    int64_t run = slots > 0 ? (b.n * per + slots - 1) / slots : kRowRunMin;
    run = run < kRowRunMin ? kRowRunMin : run > kRowRunMax ? kRowRunMax : run;
    b.run_tiles = (int32_t)run;
    const int64_t blocks = (int64_t)b.n * ((per + run - 1) / run);
    if (blocks >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
    conv_rr32_kernel<TH, 3, NS, PASS, PAIRED, MINB, ORD><<<(unsigned)blocks, kThreads, 0, st>>>(b);
    return hipGetLastError();
}

}  // namespace
// (defined in its own compilation of this file, below)
hipError_t conv_part_rr32(const ConvArgs &a, int pass, hipStream_t st);
namespace {

// Tile of the 3-channel layer with 192 outputs (the RGB input layer): rows x
// columns of output pixels per block and blocks per CU.
#ifndef HATQ_RR_TH
#define HATQ_RR_TH 2
#endif
#ifndef HATQ_RR_TW
#define HATQ_RR_TW 64
#endif
#ifndef HATQ_RR_MINB
#define HATQ_RR_MINB 2
#endif

template <int CS>
hipError_t launch_rowrun_n(const ConvArgs &a, hipStream_t st) {
    if (a.cout_pad % 192 == 0) {
        if constexpr (CS == 3) {
            const int pass = rr32_pass(a);
            if (pass >= 0) return conv_part_rr32(a, pass, st);
            const int kpass = rr32_kron_pass(a);
            if (kpass >= 0) return conv_part_rr32(a, 3 + kpass, st);
        }
        if constexpr (CS == 3)
            return with_epilogue<Epi<64, 64, 1>, Epi<64, 64, 2>, Epi<64, 64, 4>, Epi<0, 64>, Epi<0, 1>, Epi<0, 0>,
                                 Epi<64, 64>, Epi<64, 1>, Epi<64, 0>, Epi<192, 192, 5>, HATQ_KRON_EPILOGUES,
                                 HATQ_GENERIC_EPILOGUES>(
                a, [&](auto e) {
                // the requantizing pass (two transforms and the quantizer per
                // value) keeps one row group per wave: with two it spilled
                if constexpr (decltype(e)::Q == 1)
                    return launch_rowrun<HATQ_RR_TH, HATQ_RR_TW / 2, 192, CS, decltype(e), HATQ_RR_MINB>(a, st);
                else
                    return launch_rowrun<HATQ_RR_TH, HATQ_RR_TW, 192, CS, decltype(e), HATQ_RR_MINB>(a, st);
            });
        return with_epilogue<HATQ_KRON_EPILOGUES, HATQ_GENERIC_EPILOGUES>(
            a, [&](auto e) { return launch_rowrun<2, 64, 192, CS, decltype(e)>(a, st); });
    }
    if (a.cout_pad % 128 == 0)
        return with_epilogue<HATQ_S128_FIXED, HATQ_GENERIC_EPILOGUES>(
            a, [&](auto e) { return launch_rowrun<2, 64, 128, CS, decltype(e)>(a, st); });
    return with_epilogue<HATQ_GENERIC_EPILOGUES>(
        a, [&](auto e) { return launch_rowrun<2, 64, 64, CS, decltype(e)>(a, st); });
}

template <int TH, int TW, int BN, int CS, bool KRON = false>
hipError_t launch_gather(const ConvArgs &a, hipStream_t st) {
    ConvArgs b = a;
    const int64_t tiles = set_tiles(b, TH, TW, BN);
    if (tiles <= 0 || tiles >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
    auto launch = [&](auto e) {
        conv_gather_kernel<TH, TW, BN, CS, decltype(e)><<<(unsigned)tiles, kThreads, 0, st>>>(b);
        return hipGetLastError();
    };
    if constexpr (KRON) return with_epilogue<HATQ_KRON_EPILOGUES, HATQ_GENERIC_EPILOGUES>(b, launch);
    else return with_epilogue<HATQ_GENERIC_EPILOGUES>(b, launch);
}

template <int CS>
hipError_t launch_gather_n(const ConvArgs &a, hipStream_t st) {
    switch (a.cout_pad) {
        case 64: return launch_gather<8, 32, 64, CS>(a, st);
        case 128: return launch_gather<8, 32, 128, CS>(a, st);
        case 192: return launch_gather<8, 32, 192, CS, true>(a, st);
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
// The same with a wave-uniform offset added in the scalar offset field (the
// per-lane part off stays loop-invariant; an off past num_records still reads
// zeros).
__device__ __forceinline__ void dma16s(__amdgpu_buffer_rsrc_t r, int8_t *lds_dst, uint32_t off, uint32_t soff) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, HATQ_LDS_PTR(lds_dst), 16, off, soff, 0, 0);
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt");
    // s_waitcnt simm16 (gfx9): vmcnt[3:0], expcnt[6:4]=7, lgkmcnt[11:8]=15, vmcnt_hi[15:14]
    __builtin_amdgcn_s_waitcnt((N & 15) | 0x70 | 0xF00 | ((N >> 4) << 14));
}
// The same, and this wave's LDS accesses done (lgkmcnt 0).
// This wave's LDS accesses done (lgkmcnt 0), memory operations left in flight.
__device__ __forceinline__ void wait_lds() { __builtin_amdgcn_s_waitcnt(0xF | 0x70 | (3 << 14)); }
template <int N>
__device__ __forceinline__ void wait_vmcnt_lds() {
    static_assert(N >= 0 && N < 64, "vmcnt");
    __builtin_amdgcn_s_waitcnt((N & 15) | 0x70 | ((N >> 4) << 14));
}

template <int TH, int TW, int BN, int STAGES, typename E>
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
        const_cast<int8_t *>(a.wp), (short)0, (int)((int64_t)a.cout_pad * a.pack_stride), 0x00020000);

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
        b_off[j] = (uint32_t)((n0 + nn) * 64 + 16 * g);
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
        // K-blocked weights: this step's BN rows are one contiguous run
        const uint32_t woff = (uint32_t)((a.wtap[tap] * nchunks + chunk) * a.cout_pad * 64);
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
    __syncthreads();   // every wave is done with the ring; reuse it for the column factors
    float *col = reinterpret_cast<float *>(lds);
    column_factors<BN>(a, tile, col, col + BN);
    __syncthreads();
    epilogue_regs<TW, FM, FN, E>(a, acc, tile, wave * TM, lane, col, col + BN);
}

// ---------------------------------------------------------------------------
// Halo path (regular convolution, stride 2, 4 <= k <= 6, cin_p % 64 == 0): the
// input window of an 8 x 32 output tile for one 64-channel chunk, at most
// 20 x 68 pixels, stays in LDS, so each input byte crosses the L2 once per block
// instead of once per tap.  The window is split by row parity: with stride 2,
// tap row kh reads window rows 2*oh + kh, all of parity kh & 1.  Each chunk runs
// its odd-kh taps first, then its even-kh taps; while one parity half is being
// read the other half is refilled for the next phase (even half of this chunk
// during the odd taps, odd half of the next chunk during the even taps).
// Column parity is split too, so the 16 consecutive output columns a fragment
// reads are 16 consecutive 64-byte records (chunk-swizzled like the operand
// tiles: conflict-free).  Weight tiles stream through a STAGES-deep ring as in
// the pipelined path.
// ---------------------------------------------------------------------------
struct HaloGeom {
    static constexpr int TH = 8, TW = 32;
    static constexpr int HR = 10;                          // window rows per parity (k <= 6)
    static constexpr int HCC = 34;                         // window columns per parity
    static constexpr int RECS = HR * 2 * HCC;              // 64-byte records per half
    static constexpr int INSTR = (RECS + 63) / 64;         // 1 KB DMA instructions per wave per half
    static constexpr int HALF_BYTES = INSTR * 4 * 1024;
};

// Window and weight records use the operand swizzle.  With a = byte offset of
// record f (bits 0-8 of every region's base are zero), the physical address of
// chunk q is aq ^ ((aq >> 3) & 0x30) with aq = a + 16*q, so a fragment address
// is one add and two bit operations per tap.
__device__ __forceinline__ uint32_t win_addr(uint32_t aq) { return aq ^ ((aq >> 3) & 0x30u); }

// Eight waves (two per SIMD, so one wave's MFMAs run while the other waits
// on LDS), each owning one 32-pixel output row of the tile by all BN channels.
constexpr int kHaloWaves = 8;
constexpr int kHaloThreads = 64 * kHaloWaves;

// DMA block bi (1 KB) of a region of nblk >= kHaloWaves blocks, as issued by
// instruction j of a wave: blocks past the end repeat the wave's previous block
// (same bytes to the same place), so every wave issues the same number of
// instructions and the per-wave wait counts stay uniform.
__device__ __forceinline__ int halo_block(int wave, int j, int nblk) {
    const int bi = wave + kHaloWaves * j;
    return bi < nblk ? bi : bi - kHaloWaves;
}
// The same over the NW waves of one DMA role (nblk >= NW).
template <int NW>
__device__ __forceinline__ int role_block(int w, int j, int nblk) {
    const int bi = w + NW * j;
    return bi < nblk ? bi : bi - NW;
}

template <int BN, int STAGES, typename E>
__global__ void __launch_bounds__(kHaloThreads, 1) conv_halo_kernel(const ConvArgs a) {
    using G = HaloGeom;
    constexpr int TH = G::TH, TW = G::TW;
    constexpr int BM = TH * TW;
    constexpr int TM = BM / kHaloWaves;
    constexpr int FM = TM / 16;
    constexpr int FN = BN / 16;
    constexpr int B_BLK = BN / 16;                                   // 1 KB blocks per weight step
    constexpr int PER = (B_BLK + kHaloWaves - 1) / kHaloWaves;       // weight DMA instructions per wave per step
    constexpr int W_BLK = (G::RECS + 15) / 16;                       // 1 KB blocks per window half
    constexpr int HB = (W_BLK + kHaloWaves - 1) / kHaloWaves;        // window DMA instructions per wave per half
    constexpr int B_BYTES = BN * 64;
    constexpr uint32_t RING_BASE = 2 * G::HALF_BYTES;
    static_assert(BN % 64 == 0 && STAGES == 5, "tile");
    static_assert(FM == 2 && TM == TW, "one output row per wave");
    static_assert(B_BLK >= kHaloWaves && W_BLK >= kHaloWaves && W_BLK * 1024 <= G::HALF_BYTES, "DMA blocks");
    static_assert((G::HALF_BYTES & 0x1FF) == 0 && (RING_BASE & 0x1FF) == 0 && (B_BYTES & 0x1FF) == 0, "swizzle bits");
    __shared__ __attribute__((aligned(1024))) int8_t lds[2 * G::HALF_BYTES + STAGES * B_BYTES];
    int8_t *const halo = lds;
    int8_t *const bring = lds + RING_BASE;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const Tile tile = block_tile(a, xcd_logical_tile(), TH, TW, BN);
    const int n0 = tile.n0;
    const int cin_p = a.cin_p;
    const int nchunks = cin_p >> 6;
    const int k = a.k;
    const int ntap = k * k;
    const int nodd = (k >> 1) * k;                         // taps with odd kh
    const int nks = nchunks * ntap;
    const int rows_used = 2 * (TH - 1) + k, cols_used = 2 * (TW - 1) + k;
    const int ih0 = tile.gi0 * 2 + a.bah, iw0 = tile.gj0 * 2 + a.baw;

    const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int8_t *>(a.xq), (short)0, (int)((int64_t)a.n * a.h * a.w * cin_p), 0x00020000);
    const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int8_t *>(a.wp), (short)0, (int)((int64_t)a.cout_pad * a.pack_stride), 0x00020000);

    // window DMA: instruction j of this wave fills block halo_block(wave, j) of
    // a half, records 16*block + lane/4; record f = (rr*2 + cp)*HCC + cc is
    // window row 2*rr + parity, column 2*cc + cp.  Offsets exclude the chunk;
    // records outside the window or the image read zeros.
    uint32_t h_off[2][HB];
#pragma unroll
    for (int hp = 0; hp < 2; ++hp)
#pragma unroll
        for (int j = 0; j < HB; ++j) {
            const int f = 16 * halo_block(wave, j, W_BLK) + (lane >> 2);
            const int g = (lane & 3) ^ swz(f);
            const int rr = f / (2 * G::HCC), rem = f - rr * (2 * G::HCC);
            const int cp = rem / G::HCC, cc = rem - cp * G::HCC;
            const int row = 2 * rr + hp, col = 2 * cc + cp;
            const int ih = ih0 + row, iw = iw0 + col;
            const bool in = f < G::RECS && row < rows_used && col < cols_used && (unsigned)ih < (unsigned)a.h &&
                            (unsigned)iw < (unsigned)a.w;
            h_off[hp][j] = in ? (uint32_t)(((tile.nb * a.h + ih) * a.w + iw) * cin_p + 16 * g) : kOobOffset;
        }
    auto burst = [&](int hp, int chunk) {
        int8_t *dst = halo + hp * G::HALF_BYTES;
        const uint32_t coff = (uint32_t)(chunk * 64);
#pragma unroll
        for (int j = 0; j < HB; ++j)
            dma16(rx, dst + 1024 * halo_block(wave, j, W_BLK),
                  h_off[hp][j] == kOobOffset ? kOobOffset : h_off[hp][j] + coff);
    };
    uint32_t b_off[PER];
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const int nn = 16 * halo_block(wave, j, B_BLK) + (lane >> 2);
        const int g = (lane & 3) ^ swz(nn);
        b_off[j] = (uint32_t)((n0 + nn) * 64 + 16 * g);
    }

    // K-steps run chunk by chunk, odd-kh taps first, then even-kh taps.  A
    // cursor follows one step: tap index j in that order, column kw, chunk, and
    // an offset that advances with the taps (branch-free selects):
    //  * window cursors: byte offset of the tap's window records,
    //    (kh & 1)*HALF_BYTES + ((kh >> 1)*2*HCC + (kw & 1)*HCC + (kw >> 1))*64;
    //  * weight cursors: weight K-block offset ((kh*k + kw)*nchunks + chunk)*cout_pad*64.
    struct Cursor {
        int j, kw, chunk;
        uint32_t off, row_off;
    };
    const uint32_t cp64 = (uint32_t)a.cout_pad * 64u;
    const uint32_t tap_w = (uint32_t)nchunks * cp64;
    auto next_win = [&](Cursor &c) {
        const bool end_tap = c.j + 1 == ntap, end_odd = c.j + 1 == nodd, end_row = c.kw + 1 == k;
        const uint32_t in_row = c.off + ((c.kw & 1) ? (uint32_t)(64 - G::HCC * 64) : (uint32_t)(G::HCC * 64));
        const uint32_t new_row = end_tap ? (uint32_t)G::HALF_BYTES : end_odd ? 0u : c.row_off + 2u * G::HCC * 64u;
        c.off = end_row ? new_row : in_row;
        c.row_off = end_row ? new_row : c.row_off;
        c.kw = end_row ? 0 : c.kw + 1;
        c.chunk += end_tap ? 1 : 0;
        c.j = end_tap ? 0 : c.j + 1;
    };
    auto next_w = [&](Cursor &c) {
        const bool end_tap = c.j + 1 == ntap, end_odd = c.j + 1 == nodd, end_row = c.kw + 1 == k;
        const uint32_t new_row = end_tap ? (uint32_t)k * tap_w + (uint32_t)(c.chunk + 1) * cp64
                                         : end_odd ? (uint32_t)c.chunk * cp64 : c.row_off + 2u * (uint32_t)k * tap_w;
        c.off = end_row ? new_row : c.off + tap_w;
        c.row_off = end_row ? new_row : c.row_off;
        c.kw = end_row ? 0 : c.kw + 1;
        c.chunk += end_tap ? 1 : 0;
        c.j = end_tap ? 0 : c.j + 1;
    };
    // weight step of cursor c into ring slot `slot`; steps past the last one
    // read zeros into a slot no remaining step uses (uniform wait counts)
    auto issue_b = [&](const Cursor &c, int slot, bool real) {
        int8_t *sb = bring + slot * B_BYTES;
#pragma unroll
        for (int j = 0; j < PER; ++j)
            dma16(rw, sb + 1024 * halo_block(wave, j, B_BLK), real ? b_off[j] + c.off : kOobOffset);
    };

    v4i acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = v4i{0, 0, 0, 0};

    // fragment bases: this wave's pixels are output row `wave`, columns
    // 16*i + fr (A rows i = 0, 1 are 16 window records apart: same swizzle,
    // +1024 B); B column groups j are 1024 B apart
    const int fr = lane & 15, fg = lane >> 4;
    const uint32_t la0 = (uint32_t)((wave * 2 * G::HCC + fr) * 64 + 16 * fg);
    const uint32_t lb = RING_BASE + (uint32_t)(fr * 64 + 16 * (fg ^ swz(fr)));
    auto lds_v4 = [&](uint32_t addr) { return *reinterpret_cast<const v4i *>(lds + addr); };

    constexpr int RING = 4;
    static_assert(FN % RING == 0 && FN >= RING && 2 * FM <= FN, "ring");
    v4i ring[RING];
    v4i fa0[FM], fa1[FM];

    // prologue: both halves of chunk 0, weight steps 0 .. STAGES-2
    Cursor c_cur = {0, 0, 0, (uint32_t)G::HALF_BYTES, (uint32_t)G::HALF_BYTES};   // step ks (kh = 1 first)
    Cursor c_iss = {0, 0, 0, (uint32_t)k * tap_w, (uint32_t)k * tap_w};          // next weight step to issue
    burst(1, 0);
    burst(0, 0);
#pragma unroll
    for (int s = 0; s < STAGES - 1; ++s) {
        issue_b(c_iss, s, s < nks);
        next_w(c_iss);
    }
    int iss_step = STAGES - 1;
    wait_vmcnt<(STAGES - 2) * PER>();
    __builtin_amdgcn_s_barrier();
    {
        const uint32_t a0 = win_addr(la0 + c_cur.off);
        fa0[0] = lds_v4(a0);
        fa0[1] = lds_v4(a0 + 1024);
#pragma unroll
        for (int r = 0; r < RING - 1; ++r) ring[r] = lds_v4(lb + r * 1024);
    }
    Cursor c_nxt = c_cur;          // step ks+1
    next_win(c_nxt);
    int slot = 0;                  // ring slot of step ks
    // at step t's wait, since_burst = t - 1 - (step of the last window burst)
    int since_burst = 2;
    auto stage = [&](v4i (&acur)[FM], v4i (&anext)[FM]) {
        // weight steps ks and ks+1 (and the window halves they read) must have
        // landed: everything but the last two weight steps, plus a window burst
        // issued in either of the two previous steps (after weight step ks+1)
        if (since_burst <= 1) wait_vmcnt<(STAGES - 3) * PER + HB>();
        else wait_vmcnt<(STAGES - 3) * PER>();
        __builtin_amdgcn_s_barrier();
        // window refills: even half of this chunk at its first (odd) step, odd
        // half of the next chunk at this chunk's first even step
        ++since_burst;
        // (the distinct asm markers keep the two branches from being merged
        // into one path that selects its operands on every step)
        if (c_cur.j == 0 && c_cur.chunk >= 1) {
            burst(0, c_cur.chunk);
            since_burst = 0;
            asm volatile("; window refill, even rows" ::: "memory");
        } else if (c_cur.j == nodd && c_cur.chunk + 1 < nchunks) {
            burst(1, c_cur.chunk + 1);
            since_burst = 0;
            asm volatile("; window refill, odd rows" ::: "memory");
        }
        const int slot_nxt = slot == STAGES - 1 ? 0 : slot + 1;
        const int slot_iss = slot == 0 ? STAGES - 1 : slot - 1;
        issue_b(c_iss, slot_iss, iss_step < nks);
        next_w(c_iss);
        ++iss_step;
        const uint32_t bcur = lb + (uint32_t)(slot * B_BYTES), bnxt = lb + (uint32_t)(slot_nxt * B_BYTES);
        const uint32_t a0 = win_addr(la0 + c_nxt.off);
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const int jj = j + RING - 1;
            ring[jj % RING] = jj < FN ? lds_v4(bcur + jj * 1024) : lds_v4(bnxt + (jj - FN) * 1024);
            if ((j & 1) && j < 2 * FM) anext[j >> 1] = lds_v4(a0 + (j >> 1) * 1024);
#pragma unroll
            for (int i = 0; i < FM; ++i)
                acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(ring[j % RING], acur[i], acc[i][j], 0, 0, 0);
        }
        // keep the reads RING-1 fragments ahead of the MFMAs that use them
#pragma unroll
        for (int j = 0; j < FM; ++j) {
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, FM, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, FM, 0);
        }
#pragma unroll
        for (int j = 2 * FM; j < FN; ++j) {
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, FM, 0);
        }
        c_cur = c_nxt;
        next_win(c_nxt);
        slot = slot_nxt;
    };
    int ks = 0;
    for (; ks + 1 < nks; ks += 2) {
        stage(fa0, fa1);
        stage(fa1, fa0);
    }
    if (ks < nks) stage(fa0, fa1);
    wait_vmcnt<0>();   // no DMA may still be writing LDS
    __syncthreads();   // every wave is done with the window and the ring
    float *col = reinterpret_cast<float *>(lds);
    column_factors<BN>(a, tile, col, col + BN);
    __syncthreads();
    epilogue_regs<TW, FM, FN, E>(a, acc, tile, wave * TM, lane, col, col + BN);
}

// Compile-time unrolling: f(integral_constant<int, J>) for J = 0 .. N-1.
template <typename F, int... J>
__device__ __forceinline__ void unroll_seq(F &&f, std::integer_sequence<int, J...>) {
    (f(std::integral_constant<int, J>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void unroll(F &&f) {
    unroll_seq(f, std::make_integer_sequence<int, N>{});
}

// The 5 x 5 window conv with every K-step of a chunk unrolled: 25 steps per
// chunk and a 5-slot weight ring, so a step's ring slot, tap, window offset
// and wait count are compile-time constants.  The per-lane fragment addresses
// of the 15 distinct tap offsets are computed once per block, both window
// refills are issued every chunk (the odd-row refill after the last chunk
// reads zeros into rows no later step uses), and the even half of chunk 0 is
// loaded at the first step like every other chunk's.
//
// Persistent: the grid holds one block per CU and block b walks the logical
// tiles b, b + G, b + 2G, ... (G = gridDim.x, a multiple of 8, so each virtual
// block keeps the XCD of the real one and each XCD a contiguous tile range).
// The refills issued during a tile's last chunk (odd window rows and the
// first weight steps of chunk 0) fetch the next tile's data instead of zeros,
// so a tile's prologue overlaps the previous tile's last steps and epilogue.
// The weights and the per-channel scale and bias are the same for every tile
// (a launch covers one range of BN output columns, from n_base: all of them, or
// 0-191 and 192-319 of a 320-column layer in two launches); the raw scale and
// bias are staged once and each tile's column factors are formed from them and
// the sample's s_x.
template <int BN, typename E>
__global__ void __launch_bounds__(kHaloThreads, 1) conv_halo5_kernel(const ConvArgs a) {
    using G = HaloGeom;
    constexpr int K = 5, NTAP = K * K, NODD = (K >> 1) * K, SLOTS = 5;
    static_assert(NTAP % SLOTS == 0, "ring slot of a step is fixed within a chunk");
    static_assert(NTAP % 2 == 1 && NODD % 2 == 0 && SLOTS == 5, "barrier schedule");
    constexpr int TH = G::TH, TW = G::TW;
    constexpr int BM = TH * TW;
    constexpr int TM = BM / kHaloWaves;
    constexpr int FM = TM / 16;
    constexpr int FN = BN / 16;
    constexpr int B_BLK = BN / 16;
    // the DMA roles: waves 0-3 refill the weight ring, waves 4-7 the window
    // (one of each per SIMD), so a wave's vmcnt counts one kind of refill
    constexpr int RW = kHaloWaves / 2;
    constexpr int PER = (B_BLK + RW - 1) / RW;                      // weight DMAs per weight wave per step
    constexpr int W_BLK = (G::RECS + 15) / 16;
    constexpr int HB = (W_BLK + RW - 1) / RW;                       // window DMAs per window wave per half
    constexpr int B_BYTES = BN * 64;
    constexpr uint32_t RING_BASE = 2 * G::HALF_BYTES;
    static_assert(BN % 64 == 0 && FM == 2 && TM == TW, "tile");
    static_assert(B_BLK >= RW && W_BLK >= RW && W_BLK * 1024 <= G::HALF_BYTES && PER <= HB && 2 * HB <= 32,
                  "DMA blocks");
    static_assert((G::HALF_BYTES & 0x1FF) == 0 && (RING_BASE & 0x1FF) == 0 && (B_BYTES & 0x1FF) == 0, "swizzle bits");
    static_assert(G::HALF_BYTES + 1024 < 65536 && (SLOTS - 1) * B_BYTES + (FN - 1) * 1024 < 65536, "read offsets");
    static_assert(2 * (TH - 1) + K <= 2 * G::HR && 2 * (TW - 1) + K <= 2 * G::HCC, "window size");
    // one LDS object (window halves, weight ring, the tile's column factors):
    // a second one makes the compiler wait for every LDS DMA before each read
    __shared__ __attribute__((aligned(1024))) int8_t lds[2 * G::HALF_BYTES + SLOTS * B_BYTES + 4 * BN * 4];
    int8_t *const halo = lds;
    int8_t *const bring = lds + RING_BASE;
    float *const s_col = reinterpret_cast<float *>(lds + RING_BASE + SLOTS * B_BYTES);
    float *const s_raw = s_col + 2 * BN;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const bool wwave = wave < RW;               // refills the weights (else the window)
    const int ri = wwave ? wave : wave - RW;    // index within the role
    const int ntiles = a.n * a.tiles_h * a.tiles_w;   // one column range per launch
    int v = blockIdx.x;
    Tile tile = block_tile(a, xcd_tile(v, ntiles), TH, TW, BN);
    const int cin_p = a.cin_p;
    const int nchunks = cin_p >> 6;
    const int rows_used = 2 * (TH - 1) + K, cols_used = 2 * (TW - 1) + K;

    const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int8_t *>(a.xq), (short)0, (int)((int64_t)a.n * a.h * a.w * cin_p), 0x00020000);
    const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int8_t *>(a.wp), (short)0, (int)((int64_t)a.cout_pad * a.pack_stride), 0x00020000);

    // DMA offsets.  A window wave: doff[j] is the offset of its record j in the
    // even-row half (rows 2 rr), the odd-row record (2 rr + 1) one input row
    // further, and bit hp * HB + j of dmask says whether the record of half hp
    // lies in the image (else its DMA reads zeros).  A weight wave: doff[j],
    // j < PER.  One array, so the roles share the registers.
    uint32_t doff[HB];
    uint32_t dmask = 0;
    // NHWC: 64 bytes of chunk c at pixel * cin_p + 64 c; chunk-major: a plane of
    // h * w * 64 bytes per chunk (whole 128-byte lines per refill)
    const uint32_t row_stride = (uint32_t)a.w * (a.xq_c64 ? 64u : (uint32_t)cin_p);
    const uint32_t chunk_stride = a.xq_c64 ? (uint32_t)(a.h * a.w * 64) : 64u;
    auto window_offsets = [&](const Tile &t) {
        const int ih0 = t.gi0 * 2 + a.bah, iw0 = t.gj0 * 2 + a.baw;
        // the record positions afresh for each tile (a lane value the compiler
        // cannot see through): hoisted out of the tile loop, its eleven records'
        // rows and columns stayed live through the main loop and spilled in
        // the epilogue variants with the most registers
        int wl = lane;
        asm volatile("" : "+v"(wl));
        uint32_t m = 0;
#pragma unroll
        for (int j = 0; j < HB; ++j) {
            const int f = 16 * role_block<RW>(ri, j, W_BLK) + (wl >> 2);
            const int g = (wl & 3) ^ swz(f);
            const int rr = f / (2 * G::HCC), rem = f - rr * (2 * G::HCC);
            const int cp = rem / G::HCC, cc = rem - cp * G::HCC;
            const int row = 2 * rr, col = 2 * cc + cp;
            const int ih = ih0 + row, iw = iw0 + col;
            const bool cin = f < G::RECS && col < cols_used && (unsigned)iw < (unsigned)a.w;
            const bool in0 = cin && row < rows_used && (unsigned)ih < (unsigned)a.h;
            const bool in1 = cin && row + 1 < rows_used && (unsigned)(ih + 1) < (unsigned)a.h;
            // modulo 2^32 (ih may be -1 or -2 here, with its odd row inside)
            const uint32_t pix = (uint32_t)(t.nb * a.h + ih) * (uint32_t)a.w + (uint32_t)iw;
            const uint32_t off = a.xq_c64 ? (uint32_t)(t.nb * (cin_p - 64) * a.h * a.w) + pix * 64u : pix * (uint32_t)cin_p;
            doff[j] = off + 16u * g;
            m |= (in0 ? 1u << j : 0u) | (in1 ? 1u << (HB + j) : 0u);
        }
        dmask = m;
    };
    // (window waves) refill of window half hp with chunk c; zero_fill: the
    // same number of DMAs reading zeros
    auto burst = [&](int hp, int chunk) {
        int8_t *dst = halo + hp * G::HALF_BYTES;
#pragma unroll
        for (int j = 0; j < HB; ++j) {
            const uint32_t o = (dmask >> (hp * HB + j)) & 1u ? doff[j] + (hp ? row_stride : 0u) : kOobOffset;
            dma16s(rx, dst + 1024 * role_block<RW>(ri, j, W_BLK), o, (uint32_t)chunk * chunk_stride);
        }
    };
    auto zero_fill = [&](int hp) {
        int8_t *dst = halo + hp * G::HALF_BYTES;
#pragma unroll
        for (int j = 0; j < HB; ++j) dma16s(rx, dst + 1024 * role_block<RW>(ri, j, W_BLK), kOobOffset, 0u);
    };
    if (wwave) {
#pragma unroll
        for (int j = 0; j < PER; ++j) {
            const int nn = 16 * role_block<RW>(ri, j, B_BLK) + (lane >> 2);
            const int g = (lane & 3) ^ swz(nn);
            doff[j] = (uint32_t)((tile.n0 + nn) * 64 + 16 * g);
        }
    } else {
        window_offsets(tile);
    }
    const uint32_t cp64 = (uint32_t)a.cout_pad * 64u;
    const uint32_t tap_w = (uint32_t)nchunks * cp64;
    // Step j of a chunk: odd kernel rows first (kh = 1, 3), then even (0, 2, 4).
    auto step_kh = [](int j) { return j < NODD ? 1 + 2 * (j / K) : 2 * ((j - NODD) / K); };
    auto step_kw = [](int j) { return j < NODD ? j % K : (j - NODD) % K; };
    // (weight waves) weight step J of the chunk at chunk_off into its slot; or
    // zeros into it
    auto issue_b = [&](auto Jc, uint32_t chunk_off) {
        constexpr int J = decltype(Jc)::value;
        constexpr int TAP = step_kh(J) * K + step_kw(J);
        int8_t *sb = bring + (J % SLOTS) * B_BYTES;
        const uint32_t woff = (uint32_t)TAP * tap_w + chunk_off;
#pragma unroll
        for (int j = 0; j < PER; ++j) dma16s(rw, sb + 1024 * role_block<RW>(ri, j, B_BLK), doff[j], woff);
    };
    auto issue_zero = [&](auto Jc) {
        constexpr int J = decltype(Jc)::value;
        int8_t *sb = bring + (J % SLOTS) * B_BYTES;
#pragma unroll
        for (int j = 0; j < PER; ++j) dma16s(rw, sb + 1024 * role_block<RW>(ri, j, B_BLK), kOobOffset, 0u);
    };

    // per-lane A fragment addresses of the 15 window offsets (kh >> 1, kw):
    // s = (kh >> 1)*2*HCC + (kw & 1)*HCC + (kw >> 1) records; the parity half
    // and the second fragment (+16 records, same swizzle) are immediates
    const int fr = lane & 15, fg = lane >> 4;
    const uint32_t la0 = (uint32_t)((wave * 2 * G::HCC + fr) * 64 + 16 * fg);
    uint32_t pa[3 * K];
#pragma unroll
    for (int r = 0; r < 3; ++r)
#pragma unroll
        for (int kw = 0; kw < K; ++kw)
            pa[r * K + kw] = win_addr(la0 + (uint32_t)((r * 2 * G::HCC + (kw & 1) * G::HCC + (kw >> 1)) * 64));
    uint32_t lb = RING_BASE + (uint32_t)(fr * 64 + 16 * (fg ^ swz(fr)));
    // opaque bases: with known low bits the compiler would turn base + offset
    // into an or and keep one register per constant offset instead of using
    // the read's offset field
    asm volatile("" : "+v"(lb));
#pragma unroll
    for (int r = 0; r < 3 * K; ++r) asm volatile("" : "+v"(pa[r]));
    auto lds_v4 = [&](uint32_t addr) { return *reinterpret_cast<const v4i *>(lds + addr); };
    auto afrag = [&](auto Jc, int i) {
        constexpr int J = decltype(Jc)::value;
        constexpr int KH = step_kh(J % NTAP), KW = step_kw(J % NTAP);
        return lds_v4(pa[(KH >> 1) * K + KW] + (KH & 1) * G::HALF_BYTES + i * 1024);
    };
    auto bfrag = [&](auto Jc, int jj) {
        constexpr int J = decltype(Jc)::value;
        return lds_v4(lb + (J % SLOTS) * B_BYTES + jj * 1024);
    };

    v4i acc[FM][FN];

    constexpr int RING = 4;
    static_assert(FN % RING == 0 && 2 * FM <= FN, "ring");
    v4i ring[RING];
    v4i fa0[FM], fa1[FM];

    // prologue: odd half of chunk 0, weight steps 0 .. 3
    static_assert(SLOTS - 1 <= NTAP, "prologue within chunk 0");
    if (wwave)
        unroll<SLOTS - 1>([&](auto Jc) { issue_b(Jc, 0u); });
    else
        burst(1, 0);
    // the raw per-channel scale and bias, while the first DMAs are in flight
    for (int c = tid; c < BN; c += kHaloThreads) column_raw(a, tile.n0 + c, s_raw[c], s_raw[BN + c]);
    if (wwave)
        wait_vmcnt_lds<(SLOTS - 2) * PER>();
    else
        wait_vmcnt_lds<0>();
    __builtin_amdgcn_s_barrier();

  for (;;) {
    // step 0's fragments (odd window rows and weight step 0 of chunk 0 landed
    // and were published by the last barrier: the prologue's, or the last
    // step's of the previous tile, which prefetched the same values)
    fa0[0] = afrag(std::integral_constant<int, 0>{}, 0);
    fa0[1] = afrag(std::integral_constant<int, 0>{}, 1);
#pragma unroll
    for (int r = 0; r < RING - 1; ++r) ring[r] = bfrag(std::integral_constant<int, 0>{}, r);
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = v4i{0, 0, 0, 0};

    const bool first_tile = v == (int)blockIdx.x;
    for (int c = 0; c < nchunks; ++c) {
        const uint32_t coff = (uint32_t)c * cp64, coff1 = coff + cp64;
        const bool more = c + 1 < nchunks;
        // the block's next tile, if any: the refills of the last chunk fetch
        // its odd window rows and first weight steps
        const bool has_next = v + (int)gridDim.x < ntiles;
        // weight step S of this chunk (S < NTAP) or S - NTAP of the next chunk
        // (or tile), zeros past the last
        auto issue_step = [&](auto Sc) {
            constexpr int S = decltype(Sc)::value;
            if (!wwave) return;
            if constexpr (S < NTAP) {
                issue_b(std::integral_constant<int, S>{}, coff);
            } else {
                if (more || has_next) issue_b(std::integral_constant<int, S - NTAP>{}, more ? coff1 : 0u);
                else issue_zero(std::integral_constant<int, S - NTAP>{});
            }
        };
        unroll<NTAP>([&](auto Jc) {
            constexpr int J = decltype(Jc)::value;
            v4i(&acur)[FM] = (J & 1) ? fa1 : fa0;
            v4i(&anext)[FM] = (J & 1) ? fa0 : fa1;
            // One barrier per two steps (at even J; steps 24 and 0 of the
            // next chunk both have one, as a chunk has an odd number of steps).
            // At a barrier the weight waves' DMAs of the weight steps read
            // before the next barrier (up to J + 2, prefetches included; up to
            // J + 1 at J = 24) have landed; then the weight steps up to J + 4
            // are issued, whose slots were last read before this barrier.  A
            // window half is refilled right after the barrier past its last
            // read (even rows at step 0, odd rows of the next chunk at step
            // NODD) and must have landed at the barrier before its first read
            // (step NODD - 2, as step NODD - 1 prefetches step NODD's
            // fragments; step 24, which prefetches the next chunk's step 0):
            // 8 and 14 steps later.  Loads retire in issue order, so a window
            // refill in the same wave's count as the weights would have to land
            // at the weights' next wait.
            if constexpr ((J & 1) == 0) {
                if (wwave) {
                    if constexpr (J == 0) {
                        // a block's later tiles: the data of steps 0-2 was
                        // complete before the previous epilogue's stores (no
                        // wait, so the stores drain meanwhile)
                        if (c != 0 || first_tile) wait_vmcnt<PER>();
                    } else if constexpr (J == NTAP - 1) {
                        wait_vmcnt<PER>();
                    } else {
                        wait_vmcnt<0>();
                    }
                } else if constexpr (J == NODD - 2 || J == NTAP - 1) {
                    wait_vmcnt<0>();
                }
                __builtin_amdgcn_s_barrier();
                if constexpr (J == 0) {
                    issue_step(std::integral_constant<int, 4>{});
                } else if constexpr (J == NTAP - 1) {
                    issue_step(std::integral_constant<int, NTAP + 2>{});
                    issue_step(std::integral_constant<int, NTAP + 3>{});
                } else {
                    issue_step(std::integral_constant<int, J + 3>{});
                    issue_step(std::integral_constant<int, J + 4>{});
                }
                if constexpr (J == 0) {             // even rows of this chunk
                    if (!wwave) burst(0, c);
                }
                if constexpr (J == NODD) {          // odd rows of the next chunk (or tile)
                    if (!wwave) {
                        if (more) {
                            burst(1, c + 1);
                        } else if (has_next) {
                            // the even rows of this tile were fetched at step 0
                            window_offsets(block_tile(a, xcd_tile(v + (int)gridDim.x, ntiles), TH, TW, BN));
                            burst(1, 0);
                        } else {
                            zero_fill(1);
                        }
                    }
                }
            }
#pragma unroll
            for (int j = 0; j < FN; ++j) {
                const int jj = j + RING - 1;
                ring[jj % RING] = jj < FN ? bfrag(Jc, jj) : bfrag(std::integral_constant<int, J + 1>{}, jj - FN);
                if ((j & 1) && j < 2 * FM) anext[j >> 1] = afrag(std::integral_constant<int, J + 1>{}, j >> 1);
#pragma unroll
                for (int i = 0; i < FM; ++i)
                    acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(ring[j % RING], acur[i], acc[i][j], 0, 0, 0);
            }
#pragma unroll
            for (int j = 0; j < FM; ++j) {
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x008, FM, 0);
                __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
                __builtin_amdgcn_sched_group_barrier(0x008, FM, 0);
            }
#pragma unroll
            for (int j = 2 * FM; j < FN; ++j) {
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x008, FM, 0);
            }
        });
        // NTAP is odd: the next chunk's first A fragments are in fa1
#pragma unroll
        for (int i = 0; i < FM; ++i) fa0[i] = fa1[i];
    }
    {
        // the column factors and the epilogue read the arguments afresh each
        // tile (scalar loads from the kernel argument segment, through a
        // pointer the compiler cannot see through): hoisted out of the tile
        // loop they would stay live through the main loop and spill
        const __attribute__((address_space(4))) ConvArgs *kargs =
            (const __attribute__((address_space(4))) ConvArgs *)__builtin_amdgcn_kernarg_segment_ptr();
        asm volatile("" : "+s"(kargs));
        const ConvArgs &ka = *(const ConvArgs *)kargs;
        // this tile's column factors (every wave finished the previous
        // epilogue many barriers ago); the DMAs of the next tile stay in flight
        const float sxv = tile_sx_uniform(ka, tile.nb);
        for (int c = tid; c < BN; c += kHaloThreads)
            column_from_raw(ka, sxv, s_raw[c], s_raw[BN + c], s_col[c], s_col[BN + c]);
        wait_lds();
        __builtin_amdgcn_s_barrier();
        // the next tile's DMAs (its odd window rows, weight steps 0-3) complete
        // before this wave issues stores: they are then not counted behind them
        wait_vmcnt<0>();
        // the same for the lane-derived addresses and masks
        int elane = lane;
        asm volatile("" : "+v"(elane));
        epilogue_regs<TW, FM, FN, E>(ka, acc, tile, wave * TM, elane, s_col, s_col + BN);
    }
    v += gridDim.x;
    if (v >= ntiles) break;
    // a window wave's offsets are already the new tile's
    tile = block_tile(a, xcd_tile(v, ntiles), TH, TW, BN);
  }
    wait_vmcnt<0>();   // no DMA may still be writing LDS when the block ends
}

// Blocks of a persistent grid: the CU count of the current device rounded
// down to a multiple of 8 (so a virtual block keeps its XCD), or 0 if unknown.
int persistent_blocks() {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    return cus >= 8 ? cus & ~7 : 0;
}

// The arguments of the launch over samples [s0, s0 + gn) of a.
ConvArgs sample_group(const ConvArgs &a, int64_t s0, int gn) {
    ConvArgs b = a;
    b.n = gn;
    b.xq = a.xq + s0 * ((int64_t)a.h * a.w * a.cin_p);
    if (a.sx) b.sx = a.sx + s0;
    const int64_t out_per_sample = (int64_t)a.ho * a.wo * (a.mode == 0 ? a.cout_pad : a.cout);
    const int64_t elem_bytes = a.mode >= 2 ? 1 : 4;   // I8 codes, else 32-bit values
    if (a.y) b.y = (void *)((char *)a.y + s0 * out_per_sample * elem_bytes);
    if (a.next_absmax) b.next_absmax = a.next_absmax + s0;
    if (a.q_absmax) b.q_absmax = a.q_absmax + s0;
    if (a.q_scale) b.q_scale = a.q_scale + s0;
    if (a.zx) b.zx = a.zx + s0;
    b.M = (int64_t)gn * a.gh * a.gw;
    return b;
}

// split: one launch over output columns n_base .. n_base + BN - 1 of a wider
// layer (k = 5 only)
template <int BN, int STAGES, typename E>
hipError_t launch_halo(const ConvArgs &a, hipStream_t st, int n_base = 0, bool split = false) {
    static_assert(STAGES == 5, "ring");
    // keep every buffer under 2 GiB (32-bit buffer offsets, kOobOffset out of
    // range): launch over groups of whole samples
    const int64_t per_sample = (int64_t)a.h * a.w * a.cin_p;
    const int64_t group = ((int64_t)1 << 31) / per_sample;
    if (group < 1) return hipErrorInvalidValue;
    if ((int64_t)a.cout_pad * a.pack_stride >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
    if (a.sa != 2 || a.so != 1 || a.k < 4 || a.k > 6 || a.cin_p % 64) return hipErrorInvalidValue;
    const int persist = persistent_blocks();
    for (int64_t s0 = 0; s0 < a.n; s0 += group) {
        const int gn = (int)(a.n - s0 < group ? a.n - s0 : group);
        ConvArgs b = sample_group(a, s0, gn);
        int64_t tiles = set_tiles(b, HaloGeom::TH, HaloGeom::TW, BN);
        if (split) {
            if (a.k != 5 || n_base < 0 || n_base + BN > a.cout_pad) return hipErrorInvalidValue;
            b.tiles_n = 1;
            b.n_base = n_base;
            tiles = (int64_t)b.n * b.tiles_h * b.tiles_w;
        }
        if (tiles <= 0 || tiles >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
        if (a.k == 5) {
            // persistent: one block per CU (a multiple of 8), each walking tiles
            if (b.tiles_n != 1) return hipErrorInvalidValue;
            const int64_t grid = persist > 0 && persist < tiles ? persist : tiles;
            conv_halo5_kernel<BN, E><<<(unsigned)grid, kHaloThreads, 0, st>>>(b);
        } else {
            conv_halo_kernel<BN, STAGES, E><<<(unsigned)tiles, kHaloThreads, 0, st>>>(b);
        }
    }
    return hipGetLastError();
}

template <int TH, int TW, int BN, int STAGES, typename E>
hipError_t launch_pipe(const ConvArgs &a, hipStream_t st) {
    // keep every buffer under 2 GiB (32-bit buffer offsets, kOobOffset out of
    // range): launch over groups of whole samples
    const int64_t per_sample = (int64_t)a.h * a.w * a.cin_p;
    int64_t group = ((int64_t)1 << 31) / per_sample;
    if (group < 1) return hipErrorInvalidValue;
    if ((int64_t)a.cout_pad * a.pack_stride >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
    for (int64_t s0 = 0; s0 < a.n; s0 += group) {
        const int gn = (int)(a.n - s0 < group ? a.n - s0 : group);
        ConvArgs b = sample_group(a, s0, gn);
        const int64_t tiles = set_tiles(b, TH, TW, BN);
        if (tiles <= 0 || tiles >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
        conv_pipe_kernel<TH, TW, BN, STAGES, E><<<(unsigned)tiles, kThreads, 0, st>>>(b);
    }
    return hipGetLastError();
}

// Launch with the first epilogue variant of Es that matches; *hit = false,
// and nothing launched, if none does.
template <typename... Es, typename L>
hipError_t try_epilogue(const ConvArgs &a, bool *hit, L &&launch) {
    hipError_t r = hipSuccess;
    *hit = ((epi_matches<Es>(a) && (r = launch(Es{}), true)) || ...);
    return r;
}

}  // namespace

// The dispatch is spread over several compilations of this file so that the
// kernel instantiations build in parallel: HATQ_CONV_PART = k compiles part k
// only (0 is the dispatcher), and without it every part is compiled.
#ifndef HATQ_CONV_PART
#define HATQ_CONV_PART -1
#endif
#define HATQ_PART(k) (HATQ_CONV_PART < 0 || HATQ_CONV_PART == (k))

// 192 output channels, 5x5 (4x4, 6x6) stride 2: the window kernels.  The
// variant list is split in two; the order of the combined list decides.
hipError_t conv_part_halo192_a(const ConvArgs &a, bool *hit, hipStream_t st, int n_base = 0, bool split = false);
hipError_t conv_part_halo192_b(const ConvArgs &a, hipStream_t st, int n_base = 0, bool split = false);
hipError_t conv_part_halo128(const ConvArgs &a, hipStream_t st, int n_base, bool split);
hipError_t conv_part_pipe192(const ConvArgs &a, hipStream_t st);
hipError_t conv_part_pipe320(const ConvArgs &a, hipStream_t st);
hipError_t conv_part_pipe_other(const ConvArgs &a, hipStream_t st);
hipError_t conv_part_rowrun3(const ConvArgs &a, hipStream_t st);
hipError_t conv_part_rowrun_other(const ConvArgs &a, hipStream_t st);
hipError_t conv_part_gather1(const ConvArgs &a, hipStream_t st);
hipError_t conv_part_gather2(const ConvArgs &a, hipStream_t st);
hipError_t conv_part_gather3(const ConvArgs &a, hipStream_t st);
hipError_t conv_part_gather4(const ConvArgs &a, hipStream_t st);

#if HATQ_PART(1)
hipError_t conv_part_halo192_a(const ConvArgs &a, bool *hit, hipStream_t st, int n_base, bool split) {
    return try_epilogue<Epi<0, 64, 2>, Epi<0, 1, 2>, Epi<0, 0, 3>, Epi<0, 64>, Epi<0, 1>, Epi<0, 0>>(
        a, hit, [&](auto e) { return launch_halo<192, 5, decltype(e)>(a, st, n_base, split); });
}
#endif
#if HATQ_PART(2)
hipError_t conv_part_halo192_b(const ConvArgs &a, hipStream_t st, int n_base, bool split) {
    return with_epilogue<Epi<64, 64>, Epi<64, 1>, Epi<64, 0>, HATQ_KRON192_FIXED, HATQ_KRON_EPILOGUES,
                         HATQ_GENERIC_EPILOGUES>(
        a, [&](auto e) { return launch_halo<192, 5, decltype(e)>(a, st, n_base, split); });
}
#endif
#if HATQ_PART(12)
// 128 output columns of a wider 5x5 stride-2 layer (columns 192..319 of 320)
hipError_t conv_part_halo128(const ConvArgs &a, hipStream_t st, int n_base, bool split) {
    return with_epilogue<Epi<64, 0>, Epi<64, 64>, Epi<64, 1>, Epi<0, 0>, HATQ_GENERIC_EPILOGUES>(
        a, [&](auto e) { return launch_halo<128, 5, decltype(e)>(a, st, n_base, split); });
}
#endif
#if HATQ_PART(3)
hipError_t conv_part_pipe192(const ConvArgs &a, hipStream_t st) {
    return with_epilogue<Epi<0, 64>, Epi<0, 1>, Epi<0, 0>, Epi<64, 64>, Epi<64, 1>, Epi<64, 0>, HATQ_KRON_EPILOGUES,
                         HATQ_GENERIC_EPILOGUES>(
        a, [&](auto e) { return launch_pipe<8, 32, 192, 5, decltype(e)>(a, st); });
}
#endif
#if HATQ_PART(4)
hipError_t conv_part_pipe320(const ConvArgs &a, hipStream_t st) {
    return with_epilogue<Epi<0, 64>, Epi<0, 1>, Epi<0, 0>, Epi<64, 64>, Epi<64, 1>, Epi<64, 0>, HATQ_KRON320_FIXED,
                         HATQ_KRON_EPILOGUES, HATQ_GENERIC_EPILOGUES>(
        a, [&](auto e) { return launch_pipe<4, 32, 320, 5, decltype(e)>(a, st); });
}
#endif
#if HATQ_PART(5)
hipError_t conv_part_pipe_other(const ConvArgs &a, hipStream_t st) {
    switch (a.cout_pad) {
        case 128: return with_epilogue<HATQ_S128_FIXED, HATQ_GENERIC_EPILOGUES>(
                a, [&](auto e) { return launch_pipe<8, 32, 128, 5, decltype(e)>(a, st); });
        case 256: return with_epilogue<HATQ_S128_FIXED, HATQ_GENERIC_EPILOGUES>(
                a, [&](auto e) { return launch_pipe<4, 32, 256, 5, decltype(e)>(a, st); });
        default: return with_epilogue<HATQ_GENERIC_EPILOGUES>(
                a, [&](auto e) { return launch_pipe<8, 32, 64, 5, decltype(e)>(a, st); });
    }
}
#endif
#if HATQ_PART(6)
hipError_t conv_part_rowrun3(const ConvArgs &a, hipStream_t st) { return launch_rowrun_n<3>(a, st); }
#endif
#if HATQ_PART(13)
hipError_t conv_part_rr32(const ConvArgs &a, int pass, hipStream_t st) {
    // 3, 4: the absmax and codes passes with the order 192 on both sides
    if (pass == 3) return launch_rr32<HATQ_RR32_TH, 3, 0, false, HATQ_RR32_MINB_KRON, 192>(a, st);
    if (pass == 4) return launch_rr32<HATQ_RR32_TH, 3, 1, false, HATQ_RR32_MINB_KRON, 192>(a, st);
    if (pass == 2)
        return a.paired ? launch_rr32<HATQ_RR32_TH, 3, 2, true, HATQ_RR32_MINB_INT>(a, st)
                        : launch_rr32<HATQ_RR32_TH, 3, 2, false, HATQ_RR32_MINB_INT>(a, st);
    if (a.paired)
        return pass == 0 ? launch_rr32<HATQ_RR32_TH, 3, 0, true, HATQ_RR32_MINB>(a, st)
                         : launch_rr32<HATQ_RR32_TH, 3, 1, true, HATQ_RR32_MINB>(a, st);
    return pass == 0 ? launch_rr32<HATQ_RR32_TH, 3, 0, false, HATQ_RR32_MINB>(a, st)
                     : launch_rr32<HATQ_RR32_TH, 3, 1, false, HATQ_RR32_MINB>(a, st);
}
#endif
#if HATQ_PART(7)
hipError_t conv_part_rowrun_other(const ConvArgs &a, hipStream_t st) {
    switch (a.cin_p) {
        case 1: return launch_rowrun_n<1>(a, st);
        case 2: return launch_rowrun_n<2>(a, st);
        case 4: return launch_rowrun_n<4>(a, st);
        default: return hipErrorInvalidValue;
    }
}
#endif
// One part per small channel count for the gather kernel.
#define HATQ_GATHER_PART(CS)                                                                 \
    hipError_t conv_part_gather##CS(const ConvArgs &a, hipStream_t st) { return launch_gather_n<CS>(a, st); }
#if HATQ_PART(8)
HATQ_GATHER_PART(1)
#endif
#if HATQ_PART(9)
HATQ_GATHER_PART(2)
#endif
#if HATQ_PART(10)
HATQ_GATHER_PART(3)
#endif
#if HATQ_PART(11)
HATQ_GATHER_PART(4)
#endif

#if HATQ_PART(0)
hipError_t launch_conv(const ConvArgs &a, bool clear_next, hipStream_t st) {
    if (clear_next && a.next_absmax && a.next_hblock > 0)
        fill_u32_kernel<<<1, 256, 0, st>>>(reinterpret_cast<uint32_t *>(a.next_absmax), a.n, 0u);
    if (a.cin_p <= 4) {
        if (a.cin_p < 1) return hipErrorInvalidValue;
        if (a.rowrun) return a.cin_p == 3 ? conv_part_rowrun3(a, st) : conv_part_rowrun_other(a, st);
        switch (a.cin_p) {
            case 1: return conv_part_gather1(a, st);
            case 2: return conv_part_gather2(a, st);
            case 3: return conv_part_gather3(a, st);
            default: return conv_part_gather4(a, st);
        }
    }
    switch (a.cout_pad) {
        case 192:
            if (a.sa == 2 && a.so == 1 && a.k >= 4 && a.k <= 6) {
                bool hit = false;
                const hipError_t r = conv_part_halo192_a(a, &hit, st);
                return hit ? r : conv_part_halo192_b(a, st);
            }
            return conv_part_pipe192(a, st);
        case 320:
            if (a.sa == 2 && a.so == 1 && a.k == 5 && a.cin_p % 64 == 0 && !wide_needed(a)) {
                // the window kernel over columns 0..191, then 192..319 (an
                // order-320 transform spans both: the pipeline kernel's
                // 320-column tile takes those)
                bool hit = false;
                hipError_t r = conv_part_halo192_a(a, &hit, st, 0, true);
                if (!hit) r = conv_part_halo192_b(a, st, 0, true);
                if (r != hipSuccess) return r;
                return conv_part_halo128(a, st, 192, true);
            }
            return conv_part_pipe320(a, st);
        default: return conv_part_pipe_other(a, st);
    }
}
#endif

}  // namespace hatq
