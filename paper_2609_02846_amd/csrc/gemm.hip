// Decoded-operand FP4 GEMM (paper Sec. 5.1, the three products of Sec. 4.3):
//     C[m, n] = alpha * sum_k A_hat[m, k] * B_hat[n, k],  alpha = dec_a * dec_b
// with A_hat, B_hat = E2M1 value * UE5M3 block scale.  Each decoded value has
// at most 2 x 4 significant bits, its least significant bit is at least 2^-18
// and its magnitude at most 368640, so A_hat * 2^-3 is exact in fp16 (largest
// 46080, smallest step 2^-21 >= 2^-24).  The matrix cores multiply the exact
// fp16 operands exactly into fp32 and only the fp32 accumulation rounds;
// alpha * 2^6 is applied once in the epilogue (Sec. 5.2).
//
// Operands arrive contraction-contiguous (two nibbles per byte along k) with
// one scale byte per 16 k-elements; the B scale layout depends on the product:
// row blocks (wgrad), 16x16 weight tiles (fprop) or transposed weight tiles
// (dgrad).
//
// Kernel structure (gfx950, one 256-thread workgroup per CU):
//  * 256 x 256 output tile, four waves in a 2 x 2 grid, 128 x 128 per wave
//    (16 v_mfma_f32_32x32x16_f16 accumulators = 256 AccVGPRs; on gfx950 the
//    32x32 shape sustains the matrix-core peak with in-place accumulators);
//  * K advances in slices of 64.  Each thread owns one row of the A tile and
//    one row of the B tile: it loads the packed FP4 bytes and scale codes of
//    the next slice into registers while the matrix cores work on the current
//    one, decodes them to bf16 and stores them into the other half of a
//    double-buffered LDS stage (every element is decoded once per workgroup);
//  * decoding writes each UE5M3 scale s as mu * 2^E (mu = 1 + m/8 in
//    [1, 2), or 0 for code 0).  The gfx950 FP4 -> FP16 conversion applies a
//    power-of-two scale exactly (it uses only the exponent of its scale
//    operand), giving fp16(q * 2^(E-3)); one packed fp16 multiply by mu then
//    yields fp16(q * s * 2^-3) exactly.  8 nibbles cost 4 conversions and 4
//    packed multiplies; a 2 KB LDS table maps a code to (2^(E-3), mu, mu);
//  * workgroups are remapped so that each XCD runs a contiguous range of
//    tiles, walked in groups of 4 tile rows so that concurrently running
//    workgroups share A and B slices in that XCD's L2.
#include "codec.hpp"
#include "launch.hpp"

namespace ue5m3 {
namespace {

typedef __attribute__((ext_vector_type(8))) _Float16 f16x8_t;
typedef __attribute__((ext_vector_type(2))) _Float16 f16x2_t;
typedef __attribute__((ext_vector_type(16))) float f32x16_t;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4_t;

constexpr int BM = 256, BN = 256, BK = 64;
constexpr int kGemmThreads = 256;
constexpr int LDSK = BK + 8;                         // padded LDS row, bf16 elements
constexpr int kStageElems = (BM + BN) * LDSK;        // bf16 elements per stage
constexpr int kLutBytes = 256 * 8;
constexpr int kSmemBytes = 2 * kStageElems * 2 + kLutBytes;
constexpr int kXcds = 8;
constexpr int kGroupM = 4;

// Decode-table entry of UE5M3 code c: (bits of 2^(E-3), fp16 pair (mu, mu))
// with s = mu * 2^E, mu in [1, 2) a multiple of 1/8 (mu = 0 for code 0).
__device__ __forceinline__ uint2 lut_entry(uint32_t c) {
    const uint32_t e = c >> 3, m = c & 7u;
    int E;
    uint32_t mu8;                                  // mu * 8, in 8..15
    if (e == 0) {                                  // subnormal: m * 2^-17
        if (m == 0) return make_uint2(0x3F800000u, 0u);
        const int lz = __builtin_clz(m) - 28;      // shift of m to 4..7 (bit 2 set)
        mu8 = (m << lz) * 2u;                      // normalised to 8..15
        E = -17 + 2 - lz;
    } else {
        mu8 = 8u + m;
        E = (int)e - 15;
    }
    const _Float16 mu = (_Float16)((float)mu8 * 0.125f);   // exact
    uint16_t mb;
    __builtin_memcpy(&mb, &mu, 2);
    const uint32_t pow_bits = (uint32_t)(E - 3 + 127) << 23;
    return make_uint2(pow_bits, (uint32_t)mb * 0x00010001u);
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
                                            const uint2* __restrict__ lut,
                                            uint16_t* __restrict__ dst) {
    if (FULLK) v = true;
    const uint32_t code = PACKED ? (r.code[0] >> (8 * j)) & 0xFFu : r.code[j] & 0xFFu;
    const uint2 t = lut[v ? code : 0u];
    uint32_t o[8];
    decode8(v ? r.w[2 * j] : 0u, t, o);
    decode8(v ? r.w[2 * j + 1] : 0u, t, o + 4);
    uint4* d = reinterpret_cast<uint4*>(dst + 16 * j);
    d[0] = make_uint4(o[0], o[1], o[2], o[3]);
    d[1] = make_uint4(o[4], o[5], o[6], o[7]);
}

struct Frags {
    f16x8_t a[4], b[4];
};

// Fragments of k-step kk (16 k-elements) for v_mfma_f32_32x32x16_f16:
// lane l holds A[row l%32][8 k] and B[8 k][col l%32]; the k half is l/32 for
// both operands.
__device__ __forceinline__ void load_frags(Frags& f, const uint16_t* __restrict__ stage, int wm,
                                           int wn, int lane, int kk) {
    const uint16_t* la = stage + (wm * 128 + (lane & 31)) * LDSK + (lane >> 5) * 8 + kk * 16;
    const uint16_t* lb = stage + (BM + wn * 128 + (lane & 31)) * LDSK + (lane >> 5) * 8 + kk * 16;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint4 v = *reinterpret_cast<const uint4*>(la + i * 32 * LDSK);
        f.a[i] = __builtin_bit_cast(f16x8_t, u32x4_t{v.x, v.y, v.z, v.w});
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const uint4 v = *reinterpret_cast<const uint4*>(lb + j * 32 * LDSK);
        f.b[j] = __builtin_bit_cast(f16x8_t, u32x4_t{v.x, v.y, v.z, v.w});
    }
}

// The 16 MFMAs of one k-step; with DEC, the four decode blocks of one operand
// row of the next slice (r -> dst) sit between them, one per 4 MFMAs.
template <bool FULLK, bool PACKED, bool DEC>
__device__ __forceinline__ void kstep(f32x16_t (&acc)[4][4], const Frags& f, int nvalid,
                                      const RowSlice& r, const uint2* __restrict__ lut,
                                      uint16_t* __restrict__ dst) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(f.a[i], f.b[j], acc[i][j], 0, 0, 0);
        if (DEC) store_block<FULLK, PACKED>(r, i, i < nvalid, lut, dst);
    }
}

template <int BMODE, bool OUT_BF16, bool FULLK>
__global__ __launch_bounds__(kGemmThreads, 1) void gemm_fp4_kernel(
    int64_t M, int64_t N, int64_t K, int tiles_m, int tiles_n, const uint8_t* __restrict__ A,
    const uint8_t* __restrict__ As, const float* __restrict__ a_dec, const uint8_t* __restrict__ B,
    const uint8_t* __restrict__ Bs, const float* __restrict__ b_dec, void* __restrict__ C) {
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    uint16_t* stage0 = reinterpret_cast<uint16_t*>(smem);
    uint16_t* stage1 = stage0 + kStageElems;
    uint2* lut = reinterpret_cast<uint2*>(smem + 2 * kStageElems * 2);

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;

    // ---- tile index ------------------------------------------------------------
    // Workgroups are dispatched round-robin over the XCDs; remap so that each
    // XCD owns a contiguous range of tile ids, then walk tile ids in groups of
    // kGroupM tile rows (column-major inside a group) so that the ~32
    // workgroups resident on one XCD cover a kGroupM x 8 block of tiles and
    // share their A and B slices in that XCD's L2.
    const int ntiles = tiles_m * tiles_n;
    int t = blockIdx.x;
    if (ntiles % kXcds == 0) t = (t % kXcds) * (ntiles / kXcds) + t / kXcds;
    const int group_tiles = kGroupM * tiles_n;
    const int g = t / group_tiles;
    const int first_m = g * kGroupM;
    const int gm = min(tiles_m - first_m, kGroupM);
    const int rr = t - g * group_tiles;
    const int64_t m0 = (int64_t)(first_m + rr % gm) * BM;
    const int64_t n0 = (int64_t)(rr / gm) * BN;

    lut[tid] = lut_entry((uint32_t)tid);          // 256 codes, one per thread

    const int64_t kbt = K / 16;
    const int64_t nk = (K + BK - 1) / BK;
    const int64_t am = min(m0 + tid, M - 1), bn = min(n0 + tid, N - 1);
    RowSrc sa, sb;
    sa.pay = A + am * (kbt * 8);
    sa.sc = As + am * kbt;
    sa.sc_stride = 1;
    sb.pay = B + bn * (kbt * 8);
    if (BMODE == (int)BScale::Row) {
        sb.sc = Bs + bn * kbt;
        sb.sc_stride = 1;
    } else if (BMODE == (int)BScale::Tile) {
        sb.sc = Bs + (bn >> 4) * kbt;
        sb.sc_stride = 1;
    } else {
        sb.sc = Bs + (bn >> 4);
        sb.sc_stride = N >> 4;
    }
    constexpr bool kBContig = BMODE != (int)BScale::TileT;
    constexpr bool kAPacked = FULLK;
    constexpr bool kBPacked = FULLK && kBContig;
    auto nvalid = [&](int64_t s) -> int { return (int)min((int64_t)4, kbt - s * 4); };

    f32x16_t acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    if (nk > 0) {
        // Pipeline, per slice s (64 k): stage s & 1 holds slice s decoded;
        // registers (ra, rb) hold the packed bytes of slice s + 1; f0 holds
        // the k-step-0 fragments of slice s.
        //   k-step 0: 16 MFMAs + decode A row of slice s+1 -> other stage
        //   k-step 1: 16 MFMAs + decode B row of slice s+1
        //   issue the global loads of slice s+2 into (ra, rb)
        //   k-step 2: 16 MFMAs
        //   barrier (slice s+1 complete in LDS, stage s no longer read)
        //   load k-step-0 fragments of slice s+1, overlapped by
        //   k-step 3: 16 MFMAs
        // Past the end the last slice is re-loaded and re-decoded into the
        // stage nobody reads, which keeps the loop free of branches.
        const int64_t last = (nk - 1) * 4;
        RowSlice ra, rb;
        load_slice<FULLK, true>(ra, sa, 0, kbt);
        load_slice<FULLK, kBContig>(rb, sb, 0, kbt);
        __syncthreads();                              // decode table ready
        const int nv0 = nvalid(0);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            store_block<FULLK, kAPacked>(ra, j, j < nv0, lut, stage0 + tid * LDSK);
            store_block<FULLK, kBPacked>(rb, j, j < nv0, lut, stage0 + (BM + tid) * LDSK);
        }
        load_slice<FULLK, true>(ra, sa, min((int64_t)4, last), kbt);
        load_slice<FULLK, kBContig>(rb, sb, min((int64_t)4, last), kbt);
        __syncthreads();
        Frags f0, f1;
        load_frags(f0, stage0, wm, wn, lane, 0);
        for (int64_t ks = 0; ks < nk; ++ks) {
            const uint16_t* cur = (ks & 1) ? stage1 : stage0;
            uint16_t* nxt = (ks & 1) ? stage0 : stage1;
            const int nv = nvalid(ks + 1);
            load_frags(f1, cur, wm, wn, lane, 1);
            kstep<FULLK, kAPacked, true>(acc, f0, nv, ra, lut, nxt + tid * LDSK);
            __builtin_amdgcn_sched_barrier(0);
            load_frags(f0, cur, wm, wn, lane, 2);
            kstep<FULLK, kBPacked, true>(acc, f1, nv, rb, lut, nxt + (BM + tid) * LDSK);
            __builtin_amdgcn_sched_barrier(0);
            load_slice<FULLK, true>(ra, sa, min((ks + 2) * 4, last), kbt);
            load_slice<FULLK, kBContig>(rb, sb, min((ks + 2) * 4, last), kbt);
            load_frags(f1, cur, wm, wn, lane, 3);
            kstep<FULLK, false, false>(acc, f0, nv, ra, lut, nxt);
            __syncthreads();
            load_frags(f0, nxt, wm, wn, lane, 0);
            kstep<FULLK, false, false>(acc, f1, nv, ra, lut, nxt);
            __builtin_amdgcn_sched_barrier(0);
        }
    }

    // ---- epilogue: C = alpha * acc ------------------------------------------
    // 32x32 accumulator layout: lane l, register r holds
    // row 8 (r / 4) + 4 (l / 32) + r % 4, column l % 32.
    // operands were decoded as A_hat * 2^-3 and B_hat * 2^-3
    const float alpha = (a_dec[0] * b_dec[0]) * 64.0f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t n = n0 + wn * 128 + j * 32 + (lane & 31);
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int64_t m = m0 + wm * 128 + i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
                if (m < M && n < N) {
                    const float v = alpha * acc[i][j][r];
                    if (OUT_BF16) {
                        const uint32_t b = __float_as_uint(v);
                        const uint32_t rb16 = (b + 0x7FFFu + ((b >> 16) & 1u)) >> 16;
                        reinterpret_cast<uint16_t*>(C)[m * N + n] = (uint16_t)rb16;
                    } else {
                        reinterpret_cast<float*>(C)[m * N + n] = v;
                    }
                }
            }
        }
    }
}

template <int BMODE, bool OUT_BF16, bool FULLK>
hipError_t launch_one(int64_t M, int64_t N, int64_t K, const uint8_t* a, const uint8_t* as,
                      const float* ad, const uint8_t* b, const uint8_t* bs, const float* bd,
                      void* c, hipStream_t s) {
    static bool attr_set = false;
    if (!attr_set) {
        const hipError_t e = hipFuncSetAttribute(
            reinterpret_cast<const void*>(&gemm_fp4_kernel<BMODE, OUT_BF16, FULLK>),
            hipFuncAttributeMaxDynamicSharedMemorySize, kSmemBytes);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    const int tiles_m = (int)((M + BM - 1) / BM);
    const int tiles_n = (int)((N + BN - 1) / BN);
    hipLaunchKernelGGL((gemm_fp4_kernel<BMODE, OUT_BF16, FULLK>),
                       dim3((unsigned)(tiles_m * tiles_n)), dim3(kGemmThreads), kSmemBytes, s, M,
                       N, K, tiles_m, tiles_n, a, as, ad, b, bs, bd, c);
    return hipGetLastError();
}

template <int BMODE>
hipError_t launch_mode(int64_t M, int64_t N, int64_t K, const uint8_t* a, const uint8_t* as,
                       const float* ad, const uint8_t* b, const uint8_t* bs, const float* bd,
                       void* c, bool c_bf16, hipStream_t s) {
    if (K % BK == 0)
        return c_bf16 ? launch_one<BMODE, true, true>(M, N, K, a, as, ad, b, bs, bd, c, s)
                      : launch_one<BMODE, false, true>(M, N, K, a, as, ad, b, bs, bd, c, s);
    return c_bf16 ? launch_one<BMODE, true, false>(M, N, K, a, as, ad, b, bs, bd, c, s)
                  : launch_one<BMODE, false, false>(M, N, K, a, as, ad, b, bs, bd, c, s);
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
