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
// Kernel structure (gfx950, one 256-thread workgroup per CU):
//  * 256 x 256 output tile, four waves in a 2 x 2 grid, 128 x 128 per wave
//    (16 v_mfma_f32_32x32x16_bf16 accumulators = 256 AccVGPRs; on gfx950 the
//    32x32 shape sustains the matrix-core peak with in-place accumulators);
//  * K advances in slices of 64.  Each thread owns one row of the A tile and
//    one row of the B tile: it loads the packed FP4 bytes and scale codes of
//    the next slice into registers while the matrix cores work on the current
//    one, decodes them to bf16 and stores them into the other half of a
//    double-buffered LDS stage (every element is decoded once per workgroup);
//  * decoding is a byte-permute table lookup: per UE5M3 code an LDS table
//    holds the low and high bytes of bf16(q * s) for the 8 E2M1 magnitudes
//    q, so 8 nibbles become 8 bf16 with 4 table permutes, 4 interleaving
//    permutes and 3 sign operations; within each group of 8 k-elements the
//    bf16 are stored in the order 0,2,4,6,1,3,5,7 for both operands, which
//    leaves every dot product unchanged;
//  * workgroups are remapped so that each XCD runs a contiguous range of
//    tiles, ordered down tile columns so that concurrently running
//    workgroups share the B tile in that XCD's L2.
#include "codec.hpp"
#include "launch.hpp"

namespace ue5m3 {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(16))) float f32x16_t;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4_t;

constexpr int BM = 256, BN = 256, BK = 64;
constexpr int kGemmThreads = 256;
constexpr int LDSK = BK + 8;                         // padded LDS row, bf16 elements
constexpr int kStageElems = (BM + BN) * LDSK;        // bf16 elements per stage
constexpr int kLutBytes = 256 * 16;
constexpr int kSmemBytes = 2 * kStageElems * 2 + kLutBytes;
constexpr int kXcds = 8;

// bf16 bits of the E2M1 magnitude code c (0..7) times the UE5M3 scale s:
// exact, the product has at most 8 significant bits.
__device__ __forceinline__ uint32_t scaled_bf16(int c, float s) {
    const float mag[8] = {0.0f, 0.5f, 1.0f, 1.5f, 2.0f, 3.0f, 4.0f, 6.0f};
    return __float_as_uint(mag[c] * s) >> 16;
}

// Decode 8 packed nibbles x with the table entry (lo0, lo1, hi0, hi1) into
// 4 bf16x2 words holding elements (0,2), (4,6), (1,3), (5,7).
__device__ __forceinline__ void decode8(uint32_t x, const uint4& t, uint32_t* out) {
    const uint32_t e = x & 0x07070707u;                      // magnitudes 0,2,4,6
    const uint32_t o = (x >> 4) & 0x07070707u;               // magnitudes 1,3,5,7
    uint32_t he = __builtin_amdgcn_perm(t.w, t.z, e);
    const uint32_t le = __builtin_amdgcn_perm(t.y, t.x, e);
    uint32_t ho = __builtin_amdgcn_perm(t.w, t.z, o);
    const uint32_t lo = __builtin_amdgcn_perm(t.y, t.x, o);
    he |= (x << 4) & 0x80808080u;                            // sign bits of 0,2,4,6
    ho |= x & 0x80808080u;                                   // sign bits of 1,3,5,7
    out[0] = __builtin_amdgcn_perm(he, le, 0x05010400u);
    out[1] = __builtin_amdgcn_perm(he, le, 0x07030602u);
    out[2] = __builtin_amdgcn_perm(ho, lo, 0x05010400u);
    out[3] = __builtin_amdgcn_perm(ho, lo, 0x07030602u);
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
                                            const uint4* __restrict__ lut,
                                            uint16_t* __restrict__ dst) {
    if (FULLK) v = true;
    const uint32_t code = PACKED ? (r.code[0] >> (8 * j)) & 0xFFu : r.code[j] & 0xFFu;
    const uint4 t = lut[v ? code : 0u];
    uint32_t o[8];
    decode8(v ? r.w[2 * j] : 0u, t, o);
    decode8(v ? r.w[2 * j + 1] : 0u, t, o + 4);
    uint4* d = reinterpret_cast<uint4*>(dst + 16 * j);
    d[0] = make_uint4(o[0], o[1], o[2], o[3]);
    d[1] = make_uint4(o[4], o[5], o[6], o[7]);
}

struct Frags {
    bf16x8_t a[4], b[4];
};

// Fragments of k-step kk (16 k-elements) for v_mfma_f32_32x32x16_bf16:
// lane l holds A[row l%32][8 k] and B[8 k][col l%32]; the k half is l/32 for
// both operands.
__device__ __forceinline__ void load_frags(Frags& f, const uint16_t* __restrict__ la,
                                           const uint16_t* __restrict__ lb, int kk) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint4 v = *reinterpret_cast<const uint4*>(la + i * 32 * LDSK + kk * 16);
        f.a[i] = __builtin_bit_cast(bf16x8_t, u32x4_t{v.x, v.y, v.z, v.w});
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const uint4 v = *reinterpret_cast<const uint4*>(lb + j * 32 * LDSK + kk * 16);
        f.b[j] = __builtin_bit_cast(bf16x8_t, u32x4_t{v.x, v.y, v.z, v.w});
    }
}

// 16 MFMAs of one k-step; with DEC, four decode blocks of the next slice
// (blocks C0 .. C0+3 of the A row for C0 = 0, of the B row for C0 = 4) sit
// between them, one per 4 MFMAs.
template <bool FULLK, bool BPACKED, bool DEC, int C0>
__device__ __forceinline__ void kstep(f32x16_t (&acc)[4][4], const Frags& f, int nvalid,
                                      const RowSlice& ra, const RowSlice& rb,
                                      const uint4* __restrict__ lut, uint16_t* __restrict__ nxt,
                                      int tid) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[i], f.b[j], acc[i][j], 0, 0, 0);
        if (DEC) {
            if (C0 == 0) store_block<FULLK, FULLK>(ra, i, i < nvalid, lut, nxt + tid * LDSK);
            else store_block<FULLK, FULLK && BPACKED>(rb, i, i < nvalid, lut, nxt + (BM + tid) * LDSK);
        }
    }
}

// One K-slice (64 k) of matrix-core work on LDS stage `cur`.  The first two
// k-steps carry the decode of the next slice (registers ra, rb -> stage
// `nxt`); then the loads of the slice after it are issued into the freed
// registers, so that they have the last two k-steps, the barrier and the
// first k-step of the next slice to arrive.  Fragments are double-buffered
// across k-steps; the scheduling barriers keep the compiler from hoisting all
// LDS reads of the slice.
template <bool FULLK, int BMODE>
__device__ __forceinline__ void mfma_slice(f32x16_t (&acc)[4][4], const uint16_t* __restrict__ cur,
                                           int wm, int wn, int lane, int nvalid, RowSlice& ra,
                                           RowSlice& rb, const RowSrc& sa, const RowSrc& sb,
                                           int64_t kb_next, int64_t kbt,
                                           const uint4* __restrict__ lut, uint16_t* __restrict__ nxt,
                                           int tid) {
    constexpr bool kBContig = BMODE != (int)BScale::TileT;
    const uint16_t* la = cur + (wm * 128 + (lane & 31)) * LDSK + (lane >> 5) * 8;
    const uint16_t* lb = cur + (BM + wn * 128 + (lane & 31)) * LDSK + (lane >> 5) * 8;
    Frags f0, f1;
    load_frags(f0, la, lb, 0);
    load_frags(f1, la, lb, 1);
    kstep<FULLK, kBContig, true, 0>(acc, f0, nvalid, ra, rb, lut, nxt, tid);
    __builtin_amdgcn_sched_barrier(0);
    load_frags(f0, la, lb, 2);
    kstep<FULLK, kBContig, true, 4>(acc, f1, nvalid, ra, rb, lut, nxt, tid);
    __builtin_amdgcn_sched_barrier(0);
    load_slice<FULLK, true>(ra, sa, kb_next, kbt);
    load_slice<FULLK, kBContig>(rb, sb, kb_next, kbt);
    load_frags(f1, la, lb, 3);
    kstep<FULLK, kBContig, false, 0>(acc, f0, nvalid, ra, rb, lut, nxt, tid);
    __builtin_amdgcn_sched_barrier(0);
    kstep<FULLK, kBContig, false, 0>(acc, f1, nvalid, ra, rb, lut, nxt, tid);
}

template <int BMODE, bool OUT_BF16, bool FULLK>
__global__ __launch_bounds__(kGemmThreads, 1) void gemm_fp4_kernel(
    int64_t M, int64_t N, int64_t K, int tiles_m, int tiles_n, const uint8_t* __restrict__ A,
    const uint8_t* __restrict__ As, const float* __restrict__ a_dec, const uint8_t* __restrict__ B,
    const uint8_t* __restrict__ Bs, const float* __restrict__ b_dec, void* __restrict__ C) {
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    uint16_t* stage0 = reinterpret_cast<uint16_t*>(smem);
    uint16_t* stage1 = stage0 + kStageElems;
    uint4* lut = reinterpret_cast<uint4*>(smem + 2 * kStageElems * 2);

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;

    // ---- tile index: contiguous range per XCD, column-major inside ---------
    const int ntiles = tiles_m * tiles_n;
    int t = blockIdx.x;
    if (ntiles % kXcds == 0) t = (t % kXcds) * (ntiles / kXcds) + t / kXcds;
    const int64_t m0 = (int64_t)(t % tiles_m) * BM;
    const int64_t n0 = (int64_t)(t / tiles_m) * BN;

    // ---- decode table: code -> lo/hi bytes of bf16(q * s) for q = 0..7 ------
    {
        const float s = tid < 0xF8 ? ue5m3_decode((uint32_t)tid) : 0.0f;
        uint32_t lo0 = 0, lo1 = 0, hi0 = 0, hi1 = 0;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const uint32_t b0 = scaled_bf16(c, s), b1 = scaled_bf16(c + 4, s);
            lo0 |= (b0 & 0xFFu) << (8 * c);
            hi0 |= (b0 >> 8) << (8 * c);
            lo1 |= (b1 & 0xFFu) << (8 * c);
            hi1 |= (b1 >> 8) << (8 * c);
        }
        lut[tid] = make_uint4(lo0, lo1, hi0, hi1);
    }

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
    auto nvalid = [&](int64_t s) -> int { return (int)min((int64_t)4, kbt - s * 4); };

    f32x16_t acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    if (nk > 0) {
        // Slice s is decoded into LDS stage s & 1 during the matrix-core work
        // of slice s - 1; its packed bytes are loaded into (ra, rb) midway
        // through slice s - 2.
        RowSlice ra, rb;
        load_slice<FULLK, true>(ra, sa, 0, kbt);
        load_slice<FULLK, kBContig>(rb, sb, 0, kbt);
        __syncthreads();                              // decode table ready
        const int nv0 = nvalid(0);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            store_block<FULLK, FULLK>(ra, j, j < nv0, lut, stage0 + tid * LDSK);
            store_block<FULLK, FULLK && kBContig>(rb, j, j < nv0, lut, stage0 + (BM + tid) * LDSK);
        }
        const int64_t last = (nk - 1) * 4;
        load_slice<FULLK, true>(ra, sa, min((int64_t)4, last), kbt);
        load_slice<FULLK, kBContig>(rb, sb, min((int64_t)4, last), kbt);
        __syncthreads();
        // Past the end the last slice is re-loaded and re-decoded into the
        // stage nobody reads, which keeps the loop free of branches.
        for (int64_t ks = 0; ks < nk; ++ks) {
            const uint16_t* cur = (ks & 1) ? stage1 : stage0;
            uint16_t* nxt = (ks & 1) ? stage0 : stage1;
            mfma_slice<FULLK, BMODE>(acc, cur, wm, wn, lane, nvalid(ks + 1), ra, rb, sa, sb,
                                     min((ks + 2) * 4, last), kbt, lut, nxt, tid);
            __syncthreads();
        }
    }

    // ---- epilogue: C = alpha * acc ------------------------------------------
    // 32x32 accumulator layout: lane l, register r holds
    // row 8 (r / 4) + 4 (l / 32) + r % 4, column l % 32.
    const float alpha = a_dec[0] * b_dec[0];
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
