// Device-side helpers shared by the HatQ HIP kernels (gfx950 only).
//
// Fast Walsh-Hadamard butterflies.  The unnormalized Sylvester transform of
// order b = 2^L (Supplementary S-I, butterfly structure) is computed as L radix-2
// stages in ascending bit order: stage k pairs channel i with i ^ (1 << k) and
// maps (a, c) -> (a + c, a - c).  Every kernel that transforms the same data uses
// this order, so their fp32 results are bit-identical.
//
// Stages whose bit lies in the lane index use DPP lane moves and one FMA with a
// per-lane +/-1 coefficient instead of an add and a subtract.  The lane with the
// bit clear computes v + p, the lane with the bit set computes v - p = -(p - v):
// both are single correctly rounded operations, and the second carries a known
// sign flip.  The flips are tracked as a per-lane sign sigma = (-1)^(number of
// cross-lane stages in which the lane had its bit set) and removed at the end
// (or ignored where only |value| matters).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <utility>

#include "hatq_launch.h"

namespace hatq {

typedef int v4i __attribute__((ext_vector_type(4)));

// ---- DPP lane exchanges inside a 16-lane row ---------------------------------
// quad_perm [1,0,3,2]
__device__ __forceinline__ float lane_xor1(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0xB1, 0xF, 0xF, true));
}
// quad_perm [2,3,0,1]
__device__ __forceinline__ float lane_xor2(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x4E, 0xF, 0xF, true));
}
// row_half_mirror (i -> 7-i inside 8 lanes) then quad_perm [3,2,1,0] (i -> i^3):
// 7 - (i ^ 3) = i ^ 4 for i in 0..7.
__device__ __forceinline__ float lane_xor4(float v) {
    int m = __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x141, 0xF, 0xF, true);
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(m, 0x1B, 0xF, 0xF, true));
}
// row_ror:8 (i -> (i + 8) mod 16)
__device__ __forceinline__ float lane_xor8(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x128, 0xF, 0xF, true));
}

template <int MASK>
__device__ __forceinline__ float lane_xor(float v) {
    static_assert(MASK == 1 || MASK == 2 || MASK == 4 || MASK == 8, "lane mask");
    if constexpr (MASK == 1) return lane_xor1(v);
    else if constexpr (MASK == 2) return lane_xor2(v);
    else if constexpr (MASK == 4) return lane_xor4(v);
    else return lane_xor8(v);
}

// One cross-lane butterfly stage on R registers: partner lane = lane ^ MASK.
// coef = -1 on lanes with the bit set, +1 otherwise.  The partner value is the
// first factor so the DPP move folds into the fused multiply-add.
template <int MASK, int R>
__device__ __forceinline__ void cross_stage(float (&v)[R], float coef) {
#pragma unroll
    for (int r = 0; r < R; ++r) v[r] = __builtin_fmaf(lane_xor<MASK>(v[r]), coef, v[r]);
}

// One in-register butterfly stage on registers whose index bit STRIDE differs.
template <int STRIDE, int R>
__device__ __forceinline__ void reg_stage(float (&v)[R]) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
        if (r & STRIDE) continue;
        const float a = v[r], c = v[r + STRIDE];
        v[r] = a + c;
        v[r + STRIDE] = a - c;
    }
}

// ---- symmetric INT8 quantizer -----------------------------------------------
// s = fl32(A / 127), or 1 for A == 0 (IEEE division; HIP's default float
// division on gfx950 is correctly rounded).
__device__ __forceinline__ float act_scale_from_absmax(float A) {
    return A > 0.0f ? A / 127.0f : 1.0f;
}

// Magic constant 1.5 * 2^23: for |t| < 2^22, t + MAGIC rounds t to the nearest
// integer with ties to even (the hardware's default rounding of the add) and the
// low bits of the sum's encoding are that integer in two's complement.
#define HATQ_MAGIC 12582912.0f

// Exactness of the fast path: with r = fl(1/s), t = fl(v * r) differs from the
// correctly rounded quotient fl(v / s) by at most |v/s| * (3 * 2^-24 + 2^-48)
// <= 2.3e-5 for |v/s| <= 128, s a normal number.  When t lies farther than
// 0.5 - 2^-15 (2^-15 > 3.0e-5) from the nearest integer k, fl(v / s) lies
// strictly inside (k - 1/2, k + 1/2) and rne(fl(v / s)) = k.  Elements closer
// to a half-integer take the exact path, an IEEE division.
#define HATQ_NEAR_TIE (0.5f - 0x1p-15f)

// Clamp to [-127, 127].
__device__ __forceinline__ float clamp127(float t) { return __builtin_amdgcn_fmed3f(t, -127.0f, 127.0f); }

// Pack the low bytes of four 32-bit words into one word (byte 0 from a).
__device__ __forceinline__ uint32_t pack_low_bytes(uint32_t a, uint32_t b, uint32_t c, uint32_t d) {
    const uint32_t lo = __builtin_amdgcn_perm(b, a, 0x0C0C0400u);   // [a0, b0, 0, 0]
    const uint32_t hi = __builtin_amdgcn_perm(d, c, 0x0C0C0400u);   // [c0, d0, 0, 0]
    return __builtin_amdgcn_perm(hi, lo, 0x05040100u);               // [a0, b0, c0, d0]
}

// Order-preserving float max for non-negative values through 32-bit atomics.
__device__ __forceinline__ void atomic_max_nonneg(float *addr, float v) {
    atomicMax(reinterpret_cast<unsigned int *>(addr), __float_as_uint(v));
}

__device__ __forceinline__ float wave_max(float m) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
    return m;
}

// ---- Hadamard orders beyond powers of two -------------------------------------
// Paley-I matrix of order q + 1 (q prime, q = 3 mod 4): I + [[0, 1^T], [-1, Q]]
// with the Jacobsthal matrix Q[i][j] = chi(j - i), chi the quadratic character
// of F_q (chi(0) = 0).  The kernels support the Kronecker orders
// 192 = P_12 (x) H~_16 and 320 = P_20 (x) H~_16 (channel a*16 + l: the Paley
// factor on a, the Sylvester butterfly on l).
constexpr int quad_char(int a, int q) {
    a = ((a % q) + q) % q;
    if (a == 0) return 0;
    for (int x = 1; x < q; ++x)
        if ((x * x) % q == a) return 1;
    return -1;
}

constexpr int paley1_entry(int q, int i, int j) {
    const int s = i == 0 ? (j == 0 ? 0 : 1) : (j == 0 ? -1 : quad_char(j - i, q));
    return (i == j ? 1 : 0) + s;
}

// f(integral_constant<int, J>) for J = 0 .. N-1, unrolled at compile time.
template <typename F, int... J>
__device__ __forceinline__ void static_for_seq(F &&f, std::integer_sequence<int, J...>) {
    (f(std::integral_constant<int, J>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F &&f) {
    static_for_seq(f, std::make_integer_sequence<int, N>{});
}

template <int Q>
struct Paley1Table {
    int8_t s[Q + 1][Q + 1];
    constexpr Paley1Table() : s() {
        for (int i = 0; i <= Q; ++i)
            for (int j = 0; j <= Q; ++j) s[i][j] = (int8_t)paley1_entry(Q, i, j);
    }
};

template <int B>
struct ItemShape {
    static constexpr bool KRON = kron_q(B) != 0;   // P_(B/16) (x) H~_16
    static constexpr int I = B > 64 ? B : 64;      // floats per item
    static constexpr int R = I / 16;               // float4 registers per lane
    static constexpr int LOG = KRON ? 4 : B == 1 ? 0 : B == 2 ? 1 : B == 4 ? 2 : B == 8 ? 3 : B == 16 ? 4
                               : B == 32 ? 5 : B == 64 ? 6 : 7;
};

// The Paley factor of a Kronecker order on the register groups of an item:
// out[a] = sum over c, ascending, of P[a][c] * v[c] for each of the G values j
// of group c (v[G*c + j]; G = 4 in the quad and 16 x 16 MFMA layouts, 8 in the
// 32 x 32 one).  One position j at a time, so only P temporaries are live next
// to the values.
template <int Q, int R4>
__device__ __forceinline__ void paley_stage(float (&v)[R4]) {
    constexpr int P = Q + 1, G = R4 / P;   // G registers per Paley index
    static_assert(R4 == G * P && (G == 4 || G == 8), "one register group per Paley index");
    constexpr Paley1Table<Q> H{};
    // positions by a compile-time loop: with eight of them a counted loop was
    // left rolled, and its run-time register index sent v to scratch memory
    static_for<G>([&](auto jc) {
        constexpr int j = decltype(jc)::value;
        float out[P];
#pragma unroll
        for (int a = 0; a < P; ++a) {
            float acc = H.s[a][0] > 0 ? v[j] : -v[j];
#pragma unroll
            for (int c = 1; c < P; ++c) acc = H.s[a][c] > 0 ? acc + v[G * c + j] : acc - v[G * c + j];
            out[a] = acc;
        }
#pragma unroll
        for (int a = 0; a < P; ++a) v[G * a + j] = out[a];
    });
}

// The transposed factor, out[a] = sum over c, ascending, of P[c][a] * v[c]: the
// WH output restore of a Kronecker order multiplies by B^T (B^T B = m I; a
// Paley-I matrix is not symmetric).
template <int Q, int R4>
__device__ __forceinline__ void paley_stage_t(float (&v)[R4]) {
    constexpr int P = Q + 1, G = R4 / P;   // G registers per Paley index
    static_assert(R4 == G * P && (G == 4 || G == 8), "one register group per Paley index");
    constexpr Paley1Table<Q> H{};
    static_for<G>([&](auto jc) {
        constexpr int j = decltype(jc)::value;
        float out[P];
#pragma unroll
        for (int a = 0; a < P; ++a) {
            float acc = H.s[0][a] > 0 ? v[j] : -v[j];
#pragma unroll
            for (int c = 1; c < P; ++c) acc = H.s[c][a] > 0 ? acc + v[G * c + j] : acc - v[G * c + j];
            out[a] = acc;
        }
#pragma unroll
        for (int a = 0; a < P; ++a) v[G * a + j] = out[a];
    });
}

// The same on int64 values (exact, so any summation order), one register
// position j at a time to keep the temporaries small.
template <int Q, bool TRANSPOSED, int R4>
__device__ __forceinline__ void paley_stage_i64(int64_t (&v)[R4]) {
    constexpr int P = Q + 1, G = R4 / P;   // G registers per Paley index
    static_assert(R4 == G * P && (G == 4 || G == 8), "one register group per Paley index");
    constexpr Paley1Table<Q> H{};
#pragma unroll
    for (int j = 0; j < G; ++j) {
        int64_t out[P];
#pragma unroll
        for (int a = 0; a < P; ++a) {
            int64_t acc = 0;
#pragma unroll
            for (int c = 0; c < P; ++c) {
                const int sgn = TRANSPOSED ? H.s[c][a] : H.s[a][c];
                acc = sgn > 0 ? acc + v[G * c + j] : acc - v[G * c + j];
            }
            out[a] = acc;
        }
#pragma unroll
        for (int a = 0; a < P; ++a) v[G * a + j] = out[a];
    }
}

// Quad layout: one quad (4 consecutive lanes) owns an item of I = max(64, b)
// consecutive floats; lane t of the quad holds channels 16*i + 4*t + j in
// v[4*i + j].  Channel bits 0-1 (j) and 4+ (i) are inside the thread, bits 2-3
// are the quad lane.  fwht_item applies the ascending-bit butterfly of order B to
// every B-block of the item and returns sigma, the per-lane sign of the values
// held relative to the true transform.
template <int B, int R4>
__device__ __forceinline__ float fwht_item(float (&v)[R4], int t) {
    constexpr int LOG = ItemShape<B>::LOG;
    float sigma = 1.0f;
    if constexpr (LOG >= 1) reg_stage<1>(v);                 // channel bit 0
    if constexpr (LOG >= 2) reg_stage<2>(v);                 // channel bit 1
    if constexpr (LOG >= 3) {                                 // channel bit 2: lane ^ 1
        const float c = (t & 1) ? -1.0f : 1.0f;
        cross_stage<1>(v, c);
        sigma *= c;
    }
    if constexpr (LOG >= 4) {                                 // channel bit 3: lane ^ 2
        const float c = (t & 2) ? -1.0f : 1.0f;
        cross_stage<2>(v, c);
        sigma *= c;
    }
    if constexpr (LOG >= 5) reg_stage<4>(v);                 // channel bit 4: register ^ 1
    if constexpr (LOG >= 6) reg_stage<8>(v);                 // channel bit 5
    if constexpr (LOG >= 7) reg_stage<16>(v);                // channel bit 6
    if constexpr (ItemShape<B>::KRON) paley_stage<kron_q(B)>(v);   // channel bits 4+: the Paley factor
    return sigma;
}

// Fill n 32-bit words with a value (used instead of hipMemsetAsync so the
// sequence stays graph-capture friendly).
__global__ void fill_u32_kernel(uint32_t *p, int n, uint32_t v);

}  // namespace hatq
