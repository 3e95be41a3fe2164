// Device-side number formats, tensor multipliers and the Philox stream of
// the UE5M3 FP4 recipe (arXiv 2609.02846, Sec. 2-4).  Header-only, included
// by the kernel sources.  Every routine is exact integer / binary32 work; the
// files are compiled with -ffp-contract=off so that no multiply-add is fused.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ue5m3 {

constexpr float kF = 6.0f;                  // largest E2M1 magnitude (Sec. 4.2)
constexpr float kUMax = 61440.0f;           // largest UE5M3 value (eq:ue5m3max)
constexpr uint32_t kCodeMax = 0xF7u;        // its code
constexpr uint32_t kCodeOne = 0x78u;        // code of 1.0 (zero-scale rule)
constexpr float kGLimit = 0x1p110f;         // guard on the tensor multiplier

struct Multipliers {
    float S;    // T / g        : block max -> ideal scale code (eq:scale-target)
    float G;    // 6T / g       : tensor multiplier
    float dec;  // g / (6T)     : decode multiplier for the GEMM epilogue
};

// Sec. 4.2 tensor multipliers from the held amax g and target T.  A reference
// that is not positive and finite, or whose multiplier would reach 2^110
// (so that G / 2^-17 could overflow), is replaced by 1.
__device__ __forceinline__ Multipliers tensor_multipliers(float g, float T) {
    const float TF = T * kF;
    bool ok = (g > 0.0f) && (g <= 3.4028234663852886e38f);
    if (ok) {
        const float G = TF / g;
        ok = (G < kGLimit);
    }
    if (!ok) g = 1.0f;
    Multipliers m;
    m.S = T / g;
    m.G = TF / g;
    m.dec = g / TF;
    return m;
}

// UE5M3 encode of a non-negative binary32 u: nearest code, ties to the even
// code, every u above 61440 (and +inf) saturating to 0xF7.
__device__ __forceinline__ uint32_t ue5m3_encode(float u) {
    // Subnormal band [0, 2^-14): codes 0..8 are m * 2^-17, so the code is
    // RNE(u * 2^-17) -- the scaling is exact.
    const uint32_t sub = (uint32_t)__builtin_rintf(u * 0x1p17f);
    // Normal band: round the binary32 fraction to 3 bits, nearest-even, and
    // rebias the exponent from 127 to 15.  A carry propagates into the
    // exponent, which is the correct next code.
    uint32_t b = __float_as_uint(u);
    b += 0x7FFFFu + ((b >> 20) & 1u);
    const uint32_t nrm = (b >> 20) - ((127u - 15u) << 3);
    uint32_t c = (u < 0x1p-14f) ? sub : nrm;
    return (u <= kUMax) ? c : kCodeMax;
}

// UE5M3 decode of a finite code (0x00..0xF7), exact in binary32.
__device__ __forceinline__ float ue5m3_decode(uint32_t c) {
    const uint32_t e = c >> 3, m = c & 7u;
    const float sub = (float)m * 0x1p-17f;
    const float nrm = __uint_as_float(((e + 112u) << 23) | (m << 20));
    return e ? nrm : sub;
}

// ---- comparison block-scale formats (Sec. 2, Table tab:formats) ----------
// E4M3 (OCP E4M3FN: bias 7, largest finite 448 = 0x7E, 0x7F NaN, smallest
// subnormal 2^-9) encode of a non-negative binary32 u: nearest code, ties to
// the even code, every u above 448 saturating to 0x7E.
constexpr float kE4M3Max = 448.0f;
constexpr uint32_t kE4M3CodeMax = 0x7Eu;
constexpr uint32_t kE4M3CodeOne = 0x38u;
__device__ __forceinline__ uint32_t e4m3_encode(float u) {
    // subnormal band [0, 2^-6): codes 0..8 are m * 2^-9
    const uint32_t sub = (uint32_t)__builtin_rintf(u * 0x1p9f);
    // normal band: fraction rounded to 3 bits (nearest-even), exponent
    // rebased from 127 to 7; a carry lands on the next code
    uint32_t b = __float_as_uint(u);
    b += 0x7FFFFu + ((b >> 20) & 1u);
    const uint32_t nrm = (b >> 20) - ((127u - 7u) << 3);
    const uint32_t c = (u < 0x1p-6f) ? sub : nrm;
    return (u <= kE4M3Max) ? c : kE4M3CodeMax;
}

// E4M3 decode of a finite non-negative code (0x00..0x7E), exact in binary32.
__device__ __forceinline__ float e4m3_decode(uint32_t c) {
    const uint32_t e = c >> 3, m = c & 7u;
    const float sub = (float)m * 0x1p-9f;
    const float nrm = __uint_as_float(((e + 120u) << 23) | (m << 20));
    return e ? nrm : sub;
}

// E8M0 block exponent of a 32-element block from the bf16 bits of its
// largest magnitude (15-bit pattern): the OCP microscaling rule
// E = clamp(floor(log2 a) - 2, -127, 127) gives code = E + 127 =
// max(exponent field - 2, 0) for every finite bf16 a (a subnormal or zero a
// has exponent field 0 and takes code 0; the upper clamp is never reached).
__device__ __forceinline__ uint32_t e8m0_code_of_amax(uint32_t amax_bits15) {
    const int ef = (int)(amax_bits15 >> 7);
    return (uint32_t)max(ef - 2, 0);
}

// 2^-E for an E8M0 code (E = code - 127), exact: binary32 exponent field
// 254 - code, within 2..254 for every code the encoder produces (0..252).
__device__ __forceinline__ float e8m0_reciprocal(uint32_t code) {
    return __uint_as_float((254u - code) << 23);
}

// E2M1 nibble of y by stochastic rounding with the uniform 32-bit word w
// (eq:sr): between adjacent magnitudes q_lo <= |y| < q_hi round up iff
// w < ceil((|y| - q_lo) / (q_hi - q_lo) * 2^32).  |y| >= 6 gives code 7.
//  * |y| >= 1: the grid step is one unit of the 22nd binary32 fraction bit, so
//    frac * 2^32 = f22 * 2^10 with f22 the low 22 fraction bits, and the
//    event w < f22 * 2^10 is (w >> 10) < f22: exactly the carry out of the
//    low 22 bits when ~w >> 10 = 2^22 - 1 - (w >> 10) is added.  The code is
//    then the bits above, rebased: ((|y| + (~w >> 10)) >> 22) - 252.
//  * |y| < 1: step 0.5 from 0 or from 0.5; t = |y| * 2^33 (minus 2^32 from
//    0.5 up) is exact and integral at and above 2^24, so the threshold is
//    ceil(t) in integer form.
// Inputs must not be NaN (no code is specified for them).
__device__ __forceinline__ uint32_t e2m1_sr(float y, uint32_t w) {
    const uint32_t b = __float_as_uint(y);
    const uint32_t ab = b & 0x7FFFFFFFu;
    const uint32_t big = min((ab + (~w >> 10) - (252u << 22)) >> 22, 7u);
    const bool half = ab >= 0x3F000000u;                       // |y| >= 0.5
    const float t = __uint_as_float(ab) * 0x1p33f - (half ? 0x1p32f : 0.0f);
    const uint32_t thr = (uint32_t)__builtin_ceilf(t);
    const uint32_t small = (half ? 1u : 0u) + (w < thr ? 1u : 0u);
    const uint32_t c = ab >= 0x3F800000u ? big : small;
    return c | ((b >> 28) & 8u);
}

// Philox4x32-10 (Salmon et al., SC'11): four counter words, key (k0, k1),
// ten rounds of two 32x32->64 multiplies, key bumped by the Weyl constants.
// XT: truth table of the round's two three-input XORs (0x96; the
// complemented 0x69 gives ~result at no cost).
template <int XT = 0x96>
__device__ __forceinline__ uint4 philox_round(uint4 c, uint32_t k0, uint32_t k1) {
    const uint64_t p0 = (uint64_t)0xD2511F53u * c.x;
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c.z;
    const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    // three-input XORs in one instruction each
    return make_uint4(__builtin_amdgcn_bitop3_b32(hi1, c.y, k0, XT), lo1,
                      __builtin_amdgcn_bitop3_b32(hi0, c.w, k1, XT), lo0);
}

__device__ __forceinline__ uint4 philox4x32_10(uint4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        c = philox_round(c, k0, k1);
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    return c;
}

// The four SR words of source elements 4j .. 4j+3 (j = element index >> 2).
__device__ __forceinline__ uint4 sr_words4(uint64_t j, uint32_t tensor_id,
                                           uint32_t key0, uint32_t key1) {
    return philox4x32_10(make_uint4((uint32_t)j, (uint32_t)(j >> 32), tensor_id, 0u),
                         key0, key1);
}

// Their complements ~w (the operand form of the hardware SR conversion):
// the last round's XOR words come complemented from the XNOR truth table,
// the two product words take one NOT each.
__device__ __forceinline__ uint4 sr_nwords4(uint64_t j, uint32_t tensor_id,
                                            uint32_t key0, uint32_t key1) {
    uint4 c = make_uint4((uint32_t)j, (uint32_t)(j >> 32), tensor_id, 0u);
#pragma unroll
    for (int r = 0; r < 9; ++r) {
        c = philox_round(c, key0, key1);
        key0 += 0x9E3779B9u;
        key1 += 0xBB67AE85u;
    }
    c = philox_round<0x69>(c, key0, key1);
    return make_uint4(c.x, ~c.y, c.z, ~c.w);
}

// bf16 word pair -> two binary32 values (exact).
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// |x| bits of a bf16 pair as two integers (for an exact integer max).
__device__ __forceinline__ uint32_t bf16_abs_max_pair(uint32_t w) {
    const uint32_t lo = w & 0x7FFFu;
    const uint32_t hi = (w >> 16) & 0x7FFFu;
    return lo > hi ? lo : hi;
}

}  // namespace ue5m3
