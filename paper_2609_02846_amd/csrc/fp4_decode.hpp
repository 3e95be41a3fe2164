// FP4 operand decoding shared by the GEMM kernels: UE5M3 scale factors, the
// nibble -> fp16 conversion of one 8-element word, and the per-thread load
// and decode of one operand row's 64-element K slice (four blocks of 16).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ue5m3 {
namespace {

typedef __attribute__((ext_vector_type(8))) _Float16 f16x8_t;
typedef __attribute__((ext_vector_type(2))) _Float16 f16x2_t;
typedef __attribute__((ext_vector_type(16))) float f32x16_t;

// Decode factors of UE5M3 code c: the code read as an fp16 bit pattern
// shifted left by 7 (5 exponent bits with bias 15, 3 leading mantissa bits;
// code 0..7 land on the fp16 subnormals m 2^-17) is exactly its value s, so
// the factors are the power of two 2^-3 for the FP4 conversion and the fp16
// pair (s, s).  q * 2^-3 and its product with s are exact in fp16 for every
// code (|q s 2^-3| <= 46080, a multiple of 2^-24).
__device__ __forceinline__ uint2 scale_factors(uint32_t c) {
    return make_uint2(__float_as_uint(0.125f), (c << 7) | (c << 23));
}

// Decode 8 packed nibbles x (element e in bits 4e..4e+3) into 4 fp16 pairs
// (elements (0,1), (2,3), (4,5), (6,7)) of value q * s * 2^-3.
__device__ __forceinline__ void decode8(uint32_t x, const uint2& t, uint32_t* out) {
    const float p2 = __uint_as_float(t.x);
    const f16x2_t mu = __builtin_bit_cast(f16x2_t, t.y);
    const f16x2_t v0 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(x, p2, 0) * mu;
    const f16x2_t v1 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(x, p2, 1) * mu;
    const f16x2_t v2 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(x, p2, 2) * mu;
    const f16x2_t v3 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(x, p2, 3) * mu;
    out[0] = __builtin_bit_cast(uint32_t, v0);
    out[1] = __builtin_bit_cast(uint32_t, v1);
    out[2] = __builtin_bit_cast(uint32_t, v2);
    out[3] = __builtin_bit_cast(uint32_t, v3);
}

// One thread's share of a K-slice: one row of 64 k-elements (4 blocks).
// Loads go straight into these registers and nothing consumes them until the
// decode one iteration later, so no wait is placed between issue and the
// matrix-core work of the current slice.
struct RowSlice {
    uint32_t w[8];        // 4 blocks x 16 nibbles
    uint32_t code[4];     // scale code of each block (low byte)
};

// Per-thread operand row: payload row pointer and scale addressing.
struct RowSrc {
    const uint8_t* pay;   // payload row (K/2 bytes)
    const uint8_t* sc;    // scale of block 0 of this row
    int64_t sc_stride;    // byte distance between consecutive k-blocks' scales
};

// FULLK: K % 64 == 0, so every slice has 4 whole blocks, payload rows are
// 16-byte aligned and (for row/tile scales) 4 scale codes are one aligned
// word.  Otherwise blocks at or past K are clamped on load and zeroed at
// decode.  Rows past M or N are clamped to the last row: their results fall
// in output rows/columns that are never stored.
template <bool FULLK, bool SC_CONTIG>
__device__ __forceinline__ void load_slice(RowSlice& r, const RowSrc& src, int64_t kb0,
                                           int64_t kbt) {
    if (FULLK) {
        const uint4 a = *reinterpret_cast<const uint4*>(src.pay + kb0 * 8);
        const uint4 b = *reinterpret_cast<const uint4*>(src.pay + kb0 * 8 + 16);
        r.w[0] = a.x; r.w[1] = a.y; r.w[2] = a.z; r.w[3] = a.w;
        r.w[4] = b.x; r.w[5] = b.y; r.w[6] = b.z; r.w[7] = b.w;
        if (SC_CONTIG) {
            const uint32_t c4 = *reinterpret_cast<const uint32_t*>(src.sc + kb0);
            r.code[0] = c4;
            r.code[1] = c4 >> 8;
            r.code[2] = c4 >> 16;
            r.code[3] = c4 >> 24;
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) r.code[j] = src.sc[(kb0 + j) * src.sc_stride];
        }
    } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t kb = kb0 + j < kbt ? kb0 + j : kbt - 1;
            const uint2 v = *reinterpret_cast<const uint2*>(src.pay + kb * 8);
            r.w[2 * j] = v.x;
            r.w[2 * j + 1] = v.y;
            r.code[j] = src.sc[kb * src.sc_stride];
        }
    }
}

// Decode block j of a slice (16 elements) and store its 16 bf16 to LDS.
// PACKED: the four scale codes of the slice sit in the bytes of code[0]
// (one aligned word load); otherwise code[j] holds block j's code.
template <bool FULLK, bool PACKED>
__device__ __forceinline__ void store_block(const RowSlice& r, int j, bool v,
                                            uint16_t* __restrict__ dst) {
    if (FULLK) v = true;
    const uint32_t code = PACKED ? (r.code[0] >> (8 * j)) & 0xFFu : r.code[j] & 0xFFu;
    const uint2 t = scale_factors(v ? code : 0u);
    uint32_t o[8];
    decode8(v ? r.w[2 * j] : 0u, t, o);
    decode8(v ? r.w[2 * j + 1] : 0u, t, o + 4);
    uint4* d = reinterpret_cast<uint4*>(dst + 16 * j);
    d[0] = make_uint4(o[0], o[1], o[2], o[3]);
    d[1] = make_uint4(o[4], o[5], o[6], o[7]);
}

}  // namespace
}  // namespace ue5m3
