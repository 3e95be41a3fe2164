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
// one scale byte per 16 k-elements; the B scales are per row (wgrad) or per
// 16x16 weight tile (fprop, and dgrad on the transposed weight).
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
//    packed multiplies, and (2^(E-3), mu) take a few integer operations per
//    block;
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
constexpr int kSmemBytes = 2 * kStageElems * 2;
constexpr int kXcds = 8;
constexpr int kGroupM = 4;

// Decode factors of UE5M3 code c, computed arithmetically (no table, so
// decoding never waits on LDS traffic): s = mu * 2^E with
//   exponent field e >= 1: mu = 1 + m/8, E = e - 15;
//   e == 0 (s = m * 2^-17):  mu = m (an integer), E = -17.
// Returns (bits of 2^(E-3), fp16 pair (mu, mu)).  q * 2^(E-3) (the FP4
// conversion) and its product with mu are exact in fp16 for every code.
__device__ __forceinline__ uint2 scale_factors(uint32_t c) {
    const uint32_t e = (c >> 3) & 31u, m = c & 7u;
    const _Float16 mi = (_Float16)(uint16_t)m;                 // exact
    uint16_t mib;
    __builtin_memcpy(&mib, &mi, 2);
    const uint32_t mu = e ? (0x3C00u | (m << 7)) : (uint32_t)mib;
    const uint32_t pow_bits = (e ? e + 109u : 107u) << 23;
    return make_uint2(pow_bits, mu | (mu << 16));
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

// Instruction classes for the scheduling-group builtins.
constexpr int kSgValu = 0x002, kSgMfma = 0x008, kSgVmemRead = 0x020, kSgDsRead = 0x100;

// The 16 MFMAs of one k-step; with DEC, the four decode blocks of one operand
// row of the next slice (r -> dst) are interleaved with them.
template <bool FULLK, bool PACKED, bool DEC>
__device__ __forceinline__ void kstep(f32x16_t (&acc)[4][4], const Frags& f, int nvalid,
                                      const RowSlice& r, uint16_t* __restrict__ dst) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(f.a[i], f.b[j], acc[i][j], 0, 0, 0);
        if (DEC) store_block<FULLK, PACKED>(r, i, i < nvalid, dst);
    }
}

// Scheduling pattern of one k-step region: first the NDS LDS fragment reads
// for the following k-step (and NVM global loads), then the 16 MFMAs each
// followed by up to NV VALU instructions, so that the matrix cores never wait
// behind a batch of VALU work or an LDS read issued too late.
template <int NDS, int NVM, int NV>
__device__ __forceinline__ void kstep_schedule() {
    if (NVM) __builtin_amdgcn_sched_group_barrier(kSgVmemRead, NVM, 0);
    if (NDS) __builtin_amdgcn_sched_group_barrier(kSgDsRead, NDS, 0);
#pragma unroll
    for (int m = 0; m < 16; ++m) {
        __builtin_amdgcn_sched_group_barrier(kSgMfma, 1, 0);
        if (NV) __builtin_amdgcn_sched_group_barrier(kSgValu, NV, 0);
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
    } else {
        sb.sc = Bs + (bn >> 4) * kbt;
        sb.sc_stride = 1;
    }
    constexpr bool kBContig = true;
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
        const int nv0 = nvalid(0);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            store_block<FULLK, kAPacked>(ra, j, j < nv0, stage0 + tid * LDSK);
            store_block<FULLK, kBPacked>(rb, j, j < nv0, stage0 + (BM + tid) * LDSK);
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
            // k-step 0: fragments of k-step 1, MFMAs, decode of the A row
            load_frags(f1, cur, wm, wn, lane, 1);
            kstep<FULLK, kAPacked, true>(acc, f0, nv, ra, nxt + tid * LDSK);
            kstep_schedule<8, 0, 6>();
            __builtin_amdgcn_sched_barrier(0);
            // k-step 1: fragments of k-step 2, MFMAs, decode of the B row
            load_frags(f0, cur, wm, wn, lane, 2);
            kstep<FULLK, kBPacked, true>(acc, f1, nv, rb, nxt + (BM + tid) * LDSK);
            kstep_schedule<8, 0, 6>();
            __builtin_amdgcn_sched_barrier(0);
            // k-step 2: global loads of slice ks+2, fragments of k-step 3
            load_slice<FULLK, true>(ra, sa, min((ks + 2) * 4, last), kbt);
            load_slice<FULLK, kBContig>(rb, sb, min((ks + 2) * 4, last), kbt);
            load_frags(f1, cur, wm, wn, lane, 3);
            kstep<FULLK, false, false>(acc, f0, nv, ra, nxt);
            kstep_schedule<8, (FULLK ? (kBContig ? 6 : 9) : 0), 1>();
            __builtin_amdgcn_sched_barrier(0);
            __syncthreads();
            // k-step 3, overlapping the fragment reads of the next slice
            load_frags(f0, nxt, wm, wn, lane, 0);
            kstep<FULLK, false, false>(acc, f1, nv, ra, nxt);
            kstep_schedule<8, 0, 0>();
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

// ===================================================================== //
// K % 64 == 0 path: packed operands staged in LDS by direct global->LDS  //
// loads, one slice ahead, so that no register holds in-flight data.      //
// ===================================================================== //
//
// LDS (160 KB, the gfx950 maximum):
//   sF0, sF1  fp16 stages, 512 rows (256 A + 256 B) x 64 k, 128 B per row,
//             16-byte chunks XOR-swizzled by (row >> 1) & 7 so that 16
//             consecutive rows at one logical chunk hit distinct banks;
//   sP0, sP1  packed stages, 512 rows x 32 B (one slice of FP4 bytes).
// Slice x's packed bytes live in sP[x & 1] and its fp16 values in sF[x & 1].
// Per slice s (k-steps K0..K3 of 16 MFMAs each):
//   K0, K1, K2  MFMAs on sF[s&1]; decode of slice s+1 from registers
//               (A row blocks in K0 and K1, B row blocks in K1 and K2) into
//               sF[(s+1)&1];
//   wait for this thread's loads, barrier;
//   K3          read the packed rows of slice s+2 from sP[s&1] into
//               registers; start the direct loads of slice s+3 into
//               sP[(s+1)&1] and the scale words of slice s+3; read the
//               k-step-0 fragments of slice s+1; MFMAs.
// Scale words are loaded into registers (two sets, by slice parity).

constexpr int kFRow = 64;                         // fp16 per stage row
constexpr int kPRow = 32;                         // packed bytes per stage row

__device__ __forceinline__ int f_swz(int row) { return (row >> 1) & 7; }

// Decode block j (16 elements, packed words w0, w1, scale code) of one stage
// row into the swizzled fp16 stage.
__device__ __forceinline__ void decode_block_swz(uint32_t w0, uint32_t w1, uint32_t code,
                                                 uint16_t* __restrict__ frow, int sw, int j) {
    const uint2 t = scale_factors(code);
    uint32_t o[8];
    decode8(w0, t, o);
    decode8(w1, t, o + 4);
    *reinterpret_cast<uint4*>(frow + (((2 * j) ^ sw) * 8)) = make_uint4(o[0], o[1], o[2], o[3]);
    *reinterpret_cast<uint4*>(frow + (((2 * j + 1) ^ sw) * 8)) = make_uint4(o[4], o[5], o[6], o[7]);
}

__device__ __forceinline__ void load_frags_swz(Frags& f, const uint16_t* __restrict__ stage,
                                               int wm, int wn, int lane, int kk) {
    const int r = lane & 31;
    const int c = ((2 * kk + (lane >> 5)) ^ f_swz(r)) * 8;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint4 v = *reinterpret_cast<const uint4*>(stage + (wm * 128 + i * 32 + r) * kFRow + c);
        f.a[i] = __builtin_bit_cast(f16x8_t, u32x4_t{v.x, v.y, v.z, v.w});
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const uint4 v = *reinterpret_cast<const uint4*>(stage + (BM + wn * 128 + j * 32 + r) * kFRow + c);
        f.b[j] = __builtin_bit_cast(f16x8_t, u32x4_t{v.x, v.y, v.z, v.w});
    }
}

__device__ __forceinline__ void mfma16(f32x16_t (&acc)[4][4], const Frags& f) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(f.a[i], f.b[j], acc[i][j], 0, 0, 0);
}

typedef __attribute__((address_space(3))) void* lds_void_ptr;
typedef __attribute__((address_space(1))) void* glb_void_ptr;

// Direct global->LDS loads of one slice: each wave moves 64 A rows and 64 B
// rows (4 instructions of 64 lanes x 16 B).  Lane l of instruction i covers
// stage row 32 i + l / 2 (of the wave's 64), half l & 1 of its 32 bytes.
__device__ __forceinline__ void dma_slice(uint8_t* __restrict__ sp, const uint8_t* const (&src)[4],
                                          int wave, int64_t kb0) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int row0 = (q >> 1) * BM + wave * 64 + (q & 1) * 32;    // stage row of lane 0
        __builtin_amdgcn_global_load_lds((glb_void_ptr)(src[q] + kb0 * 8),
                                         (lds_void_ptr)(sp + row0 * kPRow), 16, 0, 0);
    }
}

// vmcnt(0) only (expcnt and lgkmcnt left at their maxima).
__device__ __forceinline__ void wait_vmem_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }

template <int BMODE, bool OUT_BF16>
__global__ __launch_bounds__(kGemmThreads, 1) void gemm_fp4_dma_kernel(
    int64_t M, int64_t N, int64_t K, int tiles_m, int tiles_n, const uint8_t* __restrict__ A,
    const uint8_t* __restrict__ As, const float* __restrict__ a_dec, const uint8_t* __restrict__ B,
    const uint8_t* __restrict__ Bs, const float* __restrict__ b_dec, void* __restrict__ C) {
    __shared__ __attribute__((aligned(16))) uint16_t sF0[(BM + BN) * kFRow];
    __shared__ __attribute__((aligned(16))) uint16_t sF1[(BM + BN) * kFRow];
    __shared__ __attribute__((aligned(16))) uint8_t sP0[(BM + BN) * kPRow];
    __shared__ __attribute__((aligned(16))) uint8_t sP1[(BM + BN) * kPRow];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;

    // tile index (see gemm_fp4_kernel)
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

    const int64_t kbt = K / 16;
    const int64_t rowb = kbt * 8;                 // payload row bytes
    const int64_t nk = K / BK;
    const int64_t last = (nk - 1) * 4;            // block index of the last slice

    // Direct-load sources of this lane: A rows (q = 0, 1) and B rows (q = 2, 3),
    // clamped into the matrix (clamped rows only feed discarded outputs).
    const uint8_t* dsrc[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int r = wave * 64 + (q & 1) * 32 + (lane >> 1);
        const int64_t row = (q >> 1) ? min(n0 + r, N - 1) : min(m0 + r, M - 1);
        dsrc[q] = ((q >> 1) ? B : A) + row * rowb + (lane & 1) * 16;
    }
    // Decode role: stage rows tid (A) and BM + tid (B); their scale rows.
    const int64_t am = min(m0 + tid, M - 1), bn = min(n0 + tid, N - 1);
    const uint8_t* sca = As + am * kbt;
    const uint8_t* scb = Bs + (BMODE == (int)BScale::Row ? bn : (bn >> 4)) * kbt;
    const int swa = f_swz(tid), swb = f_swz(BM + tid);
    uint16_t* fa0 = sF0 + tid * kFRow;
    uint16_t* fb0 = sF0 + (BM + tid) * kFRow;
    uint16_t* fa1 = sF1 + tid * kFRow;
    uint16_t* fb1 = sF1 + (BM + tid) * kFRow;

    f32x16_t acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    uint32_t pa[8], pb[8];                        // packed rows of the slice to decode next
    uint32_t sa0, sb0, sa1, sb1;                  // scale words, set by slice parity
    auto blk = [&](int64_t s) { return min(s * 4, last); };
    auto read_packed = [&](const uint8_t* sp) {
        const uint4 a0 = *reinterpret_cast<const uint4*>(sp + tid * kPRow);
        const uint4 a1 = *reinterpret_cast<const uint4*>(sp + tid * kPRow + 16);
        const uint4 b0 = *reinterpret_cast<const uint4*>(sp + (BM + tid) * kPRow);
        const uint4 b1 = *reinterpret_cast<const uint4*>(sp + (BM + tid) * kPRow + 16);
        pa[0] = a0.x; pa[1] = a0.y; pa[2] = a0.z; pa[3] = a0.w;
        pa[4] = a1.x; pa[5] = a1.y; pa[6] = a1.z; pa[7] = a1.w;
        pb[0] = b0.x; pb[1] = b0.y; pb[2] = b0.z; pb[3] = b0.w;
        pb[4] = b1.x; pb[5] = b1.y; pb[6] = b1.z; pb[7] = b1.w;
    };

    // ---- prologue: slices 0 and 1 staged, slice 0 decoded, slice 2 in flight
    dma_slice(sP0, dsrc, wave, 0);
    dma_slice(sP1, dsrc, wave, blk(1));
    sa0 = *reinterpret_cast<const uint32_t*>(sca);
    sb0 = *reinterpret_cast<const uint32_t*>(scb);
    sa1 = *reinterpret_cast<const uint32_t*>(sca + blk(1));
    sb1 = *reinterpret_cast<const uint32_t*>(scb + blk(1));
    wait_vmem_all();
    __syncthreads();
    read_packed(sP0);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        decode_block_swz(pa[2 * j], pa[2 * j + 1], (sa0 >> (8 * j)) & 0xFFu, fa0, swa, j);
        decode_block_swz(pb[2 * j], pb[2 * j + 1], (sb0 >> (8 * j)) & 0xFFu, fb0, swb, j);
    }
    read_packed(sP1);                             // slice 1, decoded during slice 0
    __syncthreads();                              // sF0 complete; sP0 free
    dma_slice(sP0, dsrc, wave, blk(2));
    sa0 = *reinterpret_cast<const uint32_t*>(sca + blk(2));
    sb0 = *reinterpret_cast<const uint32_t*>(scb + blk(2));
    Frags f0, f1;
    load_frags_swz(f0, sF0, wm, wn, lane, 0);

    // One slice with static buffers: P = parity of s.
    auto slice = [&](int64_t s, const uint16_t* fcur, uint16_t* fna, uint16_t* fnb,
                     const uint8_t* pcur, uint8_t* pnext, uint32_t& dsa, uint32_t& dsb) {
        // dsa/dsb: scale words of slice s+1 (decoded now), reloaded with s+3's
        // K0: fragments of k-step 1; MFMAs; A blocks 0, 1
        load_frags_swz(f1, fcur, wm, wn, lane, 1);
        mfma16(acc, f0);
        decode_block_swz(pa[0], pa[1], dsa & 0xFFu, fna, swa, 0);
        decode_block_swz(pa[2], pa[3], (dsa >> 8) & 0xFFu, fna, swa, 1);
        kstep_schedule<8, 0, 5>();
        __builtin_amdgcn_sched_barrier(0);
        // K1: fragments of k-step 2; MFMAs; A blocks 2, 3, B block 0
        load_frags_swz(f0, fcur, wm, wn, lane, 2);
        mfma16(acc, f1);
        decode_block_swz(pa[4], pa[5], (dsa >> 16) & 0xFFu, fna, swa, 2);
        decode_block_swz(pa[6], pa[7], (dsa >> 24) & 0xFFu, fna, swa, 3);
        decode_block_swz(pb[0], pb[1], dsb & 0xFFu, fnb, swb, 0);
        kstep_schedule<8, 0, 6>();
        __builtin_amdgcn_sched_barrier(0);
        // K2: fragments of k-step 3; MFMAs; B blocks 1..3
        load_frags_swz(f1, fcur, wm, wn, lane, 3);
        mfma16(acc, f0);
        decode_block_swz(pb[2], pb[3], (dsb >> 8) & 0xFFu, fnb, swb, 1);
        decode_block_swz(pb[4], pb[5], (dsb >> 16) & 0xFFu, fnb, swb, 2);
        decode_block_swz(pb[6], pb[7], (dsb >> 24) & 0xFFu, fnb, swb, 3);
        kstep_schedule<8, 0, 6>();
        __builtin_amdgcn_sched_barrier(0);
        // slice s+2 has landed in pcur (this thread's loads; then everyone's)
        wait_vmem_all();
        __syncthreads();
        // K3: packed rows of slice s+2; loads of slice s+3; fragments of the
        // next slice's k-step 0; MFMAs
        read_packed(pcur);
        dma_slice(pnext, dsrc, wave, blk(s + 3));
        dsa = *reinterpret_cast<const uint32_t*>(sca + blk(s + 3));
        dsb = *reinterpret_cast<const uint32_t*>(scb + blk(s + 3));
        load_frags_swz(f0, (fcur == sF0) ? sF1 : sF0, wm, wn, lane, 0);
        mfma16(acc, f1);
        kstep_schedule<12, 6, 0>();
        __builtin_amdgcn_sched_barrier(0);
    };
    int64_t s = 0;
    for (; s + 1 < nk; s += 2) {
        slice(s, sF0, fa1, fb1, sP0, sP1, sa1, sb1);
        slice(s + 1, sF1, fa0, fb0, sP1, sP0, sa0, sb0);
    }
    if (s < nk) slice(s, sF0, fa1, fb1, sP0, sP1, sa1, sb1);   // odd slice count
    wait_vmem_all();                              // no load outlives the kernel's LDS

    // ---- epilogue: C = alpha * acc ------------------------------------------
    const float alpha = (a_dec[0] * b_dec[0]) * 64.0f;   // operands were scaled by 2^-3
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

template <int BMODE, bool OUT_BF16>
hipError_t launch_dma(int64_t M, int64_t N, int64_t K, const uint8_t* a, const uint8_t* as,
                      const float* ad, const uint8_t* b, const uint8_t* bs, const float* bd,
                      void* c, hipStream_t s) {
    const int tiles_m = (int)((M + BM - 1) / BM);
    const int tiles_n = (int)((N + BN - 1) / BN);
    hipLaunchKernelGGL((gemm_fp4_dma_kernel<BMODE, OUT_BF16>), dim3((unsigned)(tiles_m * tiles_n)),
                       dim3(kGemmThreads), 0, s, M, N, K, tiles_m, tiles_n, a, as, ad, b, bs, bd, c);
    return hipGetLastError();
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
    if (K % BK == 0 && K > 0)
        return c_bf16 ? launch_dma<BMODE, true>(M, N, K, a, as, ad, b, bs, bd, c, s)
                      : launch_dma<BMODE, false>(M, N, K, a, as, ad, b, bs, bd, c, s);
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
    }
    return hipErrorInvalidValue;
}

}  // namespace ue5m3
