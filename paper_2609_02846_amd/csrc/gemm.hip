// Decoded-operand FP4 GEMM (paper Sec. 5.1, the three products of Sec. 4.3):
//     C[m, n] = alpha * sum_k A_hat[m, k] * B_hat[n, k],  alpha = dec_a * dec_b
// with A_hat, B_hat = E2M1 value * UE5M3 block scale.  Each decoded value has
// at most 2 x 4 significant bits and lies in [2^-18, 368640], so it is exact in
// bf16; bf16 x bf16 products are exact in fp32 and only the fp32 accumulation
// of the matrix cores rounds.  alpha is applied once in the epilogue (Sec. 5.2).
//
// Operands arrive contraction-contiguous (two nibbles per byte along k) with
// one scale byte per 16 k-elements; the B scale layout depends on the product:
// row blocks (wgrad), 16x16 weight tiles (fprop) or transposed weight tiles
// (dgrad).
//
// Kernel structure (gfx950): a 256-thread workgroup computes a BM x BN tile.
// Per BK-slice every thread loads packed FP4 + scale bytes from global memory,
// decodes its share to bf16 into LDS (each element decoded once per
// workgroup), and the four waves run v_mfma_f32_16x16x32_bf16 on LDS
// fragments.
#include "codec.hpp"
#include "launch.hpp"

namespace ue5m3 {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4_t;

constexpr int BM = 128, BN = 128, BK = 64;
constexpr int kGemmThreads = 256;
constexpr int LDSK = BK + 8;          // padded LDS row (bf16 elements)

// binary32 bits of the E2M1 magnitude code (0..7) with the sign of bit 3
__device__ __forceinline__ uint32_t e2m1_f32_bits(uint32_t nib) {
    const uint32_t mag = nib & 7u;
    uint32_t b = (mag << 22) + 0x3F000000u;            // 1.0 .. 6.0 for mag >= 2
    b = mag >= 2u ? b : (mag ? 0x3F000000u : 0u);      // 0.5 and 0
    return b | ((nib & 8u) << 28);
}

// Decode 8 nibbles (packed little-endian in p) with scale s into 8 bf16
// (4 words, element e in half e&1 of word e>>1).  q * s is exact in fp32 and
// has at most 8 significant bits, so its upper 16 bits are its bf16 value.
__device__ __forceinline__ void decode8(uint32_t p, float s, uint32_t* out) {
#pragma unroll
    for (int e = 0; e < 8; e += 2) {
        const float v0 = __uint_as_float(e2m1_f32_bits(p >> (4 * e))) * s;
        const float v1 = __uint_as_float(e2m1_f32_bits(p >> (4 * e + 4))) * s;
        out[e >> 1] = (__float_as_uint(v0) >> 16) | (__float_as_uint(v1) & 0xFFFF0000u);
    }
}

template <int BMODE, bool OUT_BF16>
__global__ __launch_bounds__(kGemmThreads) void gemm_fp4_kernel(
    int64_t M, int64_t N, int64_t K, const uint8_t* __restrict__ A, const uint8_t* __restrict__ As,
    const float* __restrict__ a_dec, const uint8_t* __restrict__ B,
    const uint8_t* __restrict__ Bs, const float* __restrict__ b_dec, void* __restrict__ C) {
    __shared__ __attribute__((aligned(16))) uint16_t lds_a[BM * LDSK];
    __shared__ __attribute__((aligned(16))) uint16_t lds_b[BN * LDSK];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;           // 2 x 2 waves, 64 x 64 each
    const int64_t m0 = (int64_t)blockIdx.y * BM;
    const int64_t n0 = (int64_t)blockIdx.x * BN;
    const int64_t ldp = K / 2;                          // payload row stride (bytes)
    const int64_t kb_total = K / 16;                    // scale blocks per row

    // loader role: row (tid >> 1) of the A and B tiles, k-half (tid & 1)
    const int lrow = tid >> 1;
    const int lhalf = tid & 1;
    const int64_t am = m0 + lrow, bn = n0 + lrow;
    const bool a_ok = am < M, b_ok = bn < N;

    f32x4_t acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    for (int64_t k0 = 0; k0 < K; k0 += BK) {
        // ---- global -> registers: 2 blocks of 16 for A and B --------------
        uint32_t apk[4] = {0u, 0u, 0u, 0u}, bpk[4] = {0u, 0u, 0u, 0u};
        float asc[2] = {0.f, 0.f}, bsc[2] = {0.f, 0.f};
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int64_t kb = k0 / 16 + lhalf * 2 + j;      // 16-block index along k
            if (kb < kb_total) {
                if (a_ok) {
                    const uint2 t = *reinterpret_cast<const uint2*>(A + am * ldp + kb * 8);
                    apk[2 * j] = t.x;
                    apk[2 * j + 1] = t.y;
                    asc[j] = ue5m3_decode(As[am * kb_total + kb]);
                }
                if (b_ok) {
                    const uint2 t = *reinterpret_cast<const uint2*>(B + bn * ldp + kb * 8);
                    bpk[2 * j] = t.x;
                    bpk[2 * j + 1] = t.y;
                    uint32_t code;
                    if (BMODE == (int)BScale::Row) code = Bs[bn * kb_total + kb];
                    else if (BMODE == (int)BScale::Tile) code = Bs[(bn >> 4) * kb_total + kb];
                    else code = Bs[kb * (N >> 4) + (bn >> 4)];
                    bsc[j] = ue5m3_decode(code);
                }
            }
        }
        // ---- decode to bf16 ------------------------------------------------
        uint32_t adec[16], bdec[16];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            decode8(apk[q], asc[q >> 1], adec + 4 * q);
            decode8(bpk[q], bsc[q >> 1], bdec + 4 * q);
        }
        __syncthreads();                                  // previous slice consumed
        {
            uint32_t* pa = reinterpret_cast<uint32_t*>(lds_a + lrow * LDSK + lhalf * 32);
            uint32_t* pb = reinterpret_cast<uint32_t*>(lds_b + lrow * LDSK + lhalf * 32);
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                reinterpret_cast<uint4*>(pa)[q] =
                    make_uint4(adec[4 * q], adec[4 * q + 1], adec[4 * q + 2], adec[4 * q + 3]);
                reinterpret_cast<uint4*>(pb)[q] =
                    make_uint4(bdec[4 * q], bdec[4 * q + 1], bdec[4 * q + 2], bdec[4 * q + 3]);
            }
        }
        __syncthreads();
        // ---- MFMA on the slice -------------------------------------------
#pragma unroll
        for (int kk = 0; kk < BK / 32; ++kk) {
            const int kof = kk * 32 + (lane >> 4) * 8;
            bf16x8_t af[4], bfr[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const uint4 t = *reinterpret_cast<const uint4*>(
                    lds_a + (wm * 64 + i * 16 + (lane & 15)) * LDSK + kof);
                af[i] = __builtin_bit_cast(bf16x8_t, u32x4_t{t.x, t.y, t.z, t.w});
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const uint4 t = *reinterpret_cast<const uint4*>(
                    lds_b + (wn * 64 + j * 16 + (lane & 15)) * LDSK + kof);
                bfr[j] = __builtin_bit_cast(bf16x8_t, u32x4_t{t.x, t.y, t.z, t.w});
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
        }
    }

    // ---- epilogue: C = alpha * acc -------------------------------------
    const float alpha = a_dec[0] * b_dec[0];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t n = n0 + wn * 64 + j * 16 + (lane & 15);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int64_t m = m0 + wm * 64 + i * 16 + (lane >> 4) * 4 + r;
                if (m < M && n < N) {
                    const float v = alpha * acc[i][j][r];
                    if (OUT_BF16) {
                        const uint32_t b = __float_as_uint(v);
                        const uint32_t rb = (b + 0x7FFFu + ((b >> 16) & 1u)) >> 16;
                        reinterpret_cast<uint16_t*>(C)[m * N + n] = (uint16_t)rb;
                    } else {
                        reinterpret_cast<float*>(C)[m * N + n] = v;
                    }
                }
            }
        }
    }
}

template <int BMODE>
hipError_t launch_mode(int64_t M, int64_t N, int64_t K, const uint8_t* a, const uint8_t* as,
                       const float* ad, const uint8_t* b, const uint8_t* bs, const float* bd,
                       void* c, bool c_bf16, hipStream_t s) {
    const dim3 grid((unsigned)((N + BN - 1) / BN), (unsigned)((M + BM - 1) / BM));
    if (c_bf16)
        hipLaunchKernelGGL((gemm_fp4_kernel<BMODE, true>), grid, dim3(kGemmThreads), 0, s, M, N, K,
                           a, as, ad, b, bs, bd, c);
    else
        hipLaunchKernelGGL((gemm_fp4_kernel<BMODE, false>), grid, dim3(kGemmThreads), 0, s, M, N, K,
                           a, as, ad, b, bs, bd, c);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm(BScale bmode, int64_t M, int64_t N, int64_t K, const uint8_t* a,
                       const uint8_t* a_scales, const float* a_dec, const uint8_t* b,
                       const uint8_t* b_scales, const float* b_dec, void* c, bool c_bf16,
                       hipStream_t s) {
    if (M == 0 || N == 0) return hipSuccess;
    switch (bmode) {
        case BScale::Row:
            return launch_mode<(int)BScale::Row>(M, N, K, a, a_scales, a_dec, b, b_scales, b_dec, c, c_bf16, s);
        case BScale::Tile:
            return launch_mode<(int)BScale::Tile>(M, N, K, a, a_scales, a_dec, b, b_scales, b_dec, c, c_bf16, s);
        case BScale::TileT:
            return launch_mode<(int)BScale::TileT>(M, N, K, a, a_scales, a_dec, b, b_scales, b_dec, c, c_bf16, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace ue5m3
