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
// Kernels (gfx950, one 256-thread workgroup per CU, 256 x 256 output tiles,
// four waves of 128 x 128 in a 2 x 2 grid, 16 v_mfma_f32_32x32x16_f16
// accumulators per wave = all 256 AccVGPRs):
//  * K % 256 == 0, operands and C below 2^31 bytes: gemm_fp4_reg_kernel,
//    persistent; packed FP4 rows and scale codes staged in LDS by direct
//    loads four 64-k slices at a time, each wave decoding its own fragments
//    in registers (no fp16 copy through LDS);
//  * K % 64 == 0: gemm_fp4_dma_kernel, packed slices staged by direct loads
//    and decoded once per workgroup into a double-buffered fp16 LDS stage;
//  * any K % 16 == 0: gemm_fp4_kernel, the same with register-staged loads.
// Decoding writes each UE5M3 scale s as mu * 2^E (mu = 1 + m/8 in [1, 2), or
// 0 for code 0) or reads the code as an fp16 bit pattern (c << 7 is its
// value).  The gfx950 FP4 -> FP16 conversion applies a power-of-two scale
// exactly (it uses only the exponent of its scale operand), giving
// fp16(q * 2^(E-3)); one packed fp16 multiply by mu (or by the code's value
// after a 2^-3 conversion) then yields fp16(q * s * 2^-3) exactly.
// Workgroups are remapped so that each XCD runs a contiguous range of tiles,
// walked in groups of 4 tile rows so that concurrently running workgroups
// share A and B slices in that XCD's L2.
#include "codec.hpp"
#include "fp4_decode.hpp"
#include "launch.hpp"

#include <atomic>
#include <type_traits>

namespace ue5m3 {
namespace {

typedef __attribute__((ext_vector_type(4))) uint32_t u32x4_t;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;

constexpr int BM = 256, BN = 256, BK = 64;
constexpr int kGemmThreads = 256;
constexpr int LDSK = BK + 8;                         // padded LDS row, bf16 elements
constexpr int kStageElems = (BM + BN) * LDSK;        // bf16 elements per stage
constexpr int kSmemBytes = 2 * kStageElems * 2;
constexpr int kXcds = 8;
constexpr int kGroupM = 4;

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
    const uint8_t* __restrict__ Bs, const float* __restrict__ b_dec, void* __restrict__ C, float amul) {
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
    const float alpha = (a_dec[0] * b_dec[0]) * amul;
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

// The same products issued as B x A^T: accumulator (i, j) then holds the
// transposed 32 x 32 block, so that each lane owns runs of 4 adjacent output
// columns (element e of lane l: row l%32, column 8(e/4) + 4(l/32) + e%4).
__device__ __forceinline__ void mfma16_t(f32x16_t (&acc)[4][4], const Frags& f) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(f.b[j], f.a[i], acc[i][j], 0, 0, 0);
}

// Two floats to two bf16 (round to nearest even), packed low-first.
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
    typedef __attribute__((ext_vector_type(2))) float f32x2_t;
    typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;
    const f32x2_t v = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
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
    const uint8_t* __restrict__ Bs, const float* __restrict__ b_dec, void* __restrict__ C, float amul) {
    __shared__ __attribute__((aligned(16))) uint16_t sF0[(BM + BN) * kFRow];
    __shared__ __attribute__((aligned(16))) uint16_t sF1[(BM + BN) * kFRow];
    __shared__ __attribute__((aligned(16))) uint8_t sP0[(BM + BN) * kPRow];
    __shared__ __attribute__((aligned(16))) uint8_t sP1[(BM + BN) * kPRow];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;

    // tile index (see tile_origin)
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
    const float alpha = (a_dec[0] * b_dec[0]) * amul;   // operands were scaled by 2^-3
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
                      void* c, float amul, hipStream_t s) {
    const int tiles_m = (int)((M + BM - 1) / BM);
    const int tiles_n = (int)((N + BN - 1) / BN);
    hipLaunchKernelGGL((gemm_fp4_dma_kernel<BMODE, OUT_BF16>), dim3((unsigned)(tiles_m * tiles_n)),
                       dim3(kGemmThreads), 0, s, M, N, K, tiles_m, tiles_n, a, as, ad, b, bs, bd, c, amul);
    return hipGetLastError();
}

// ===================================================================== //
// K % 256 == 0 path: decode straight into MFMA fragments.               //
// ===================================================================== //
//
// The workgroup stages its 256 A rows and 256 B rows in LDS four K slices at
// a time (256 k: 128 payload bytes and 16 scale bytes per row), double
// buffered and filled by direct global->LDS loads, with one barrier per four
// slices.  Each wave then decodes its fragments itself: no fp16 copy of the
// operands goes through LDS.
//
// For k-step kk (0..3) of slice sl, lane l of the 32x32x16 MFMA supplies 8
// k-elements of row l % 32: half h = l / 32 takes payload word 4h + kk of
// the row's 32 bytes of that slice (k = 64 sl + 32h + 8kk .. + 7).  The k
// order inside a slice is thus permuted, identically for A and B, which the
// sum over k does not see.  That word's block scale is code 2h + kk/2 of the
// row's scale word for the slice.
//
// A UE5M3 code c read as an fp16 bit pattern, c << 7, is exactly its value
// (5 exponent bits with bias 15, 3 leading mantissa bits, subnormals
// included; codes above 0xF7 are not valid encodings).  The decode is
// therefore two exact steps: the hardware FP4 -> FP16 conversion with the
// power-of-two scale 2^-3, then an fp16 multiply by the code's value.  The
// product q * s * 2^-3 never exceeds 6 * 61440 / 8 = 46080 and is a multiple
// of 2^-24, so it is representable in fp16.
//
// A stage row is 128 B = 8 chunks of 16 B; chunk c of stage row x sits at
// position c ^ (x & 7), so that the 8 lanes the LDS serves together hit 8
// different bank groups.

constexpr int kSupK = 4;                                  // slices per stage
constexpr int kSupRows = BM + BN;                         // 512 stage rows
constexpr int kSupRowBytes = kSupK * 32;                  // 128
constexpr int kSupPayload = kSupRows * kSupRowBytes;      // 64 KB
constexpr int kSupScales = kSupRows * kSupK * 4;          // 8 KB
constexpr int kSupPayLoads = kSupPayload / 1024 / 4;      // 16 payload loads per wave
constexpr int kSupScLoads = kSupScales / 1024 / 4;        // 2 scale loads per wave
constexpr int kSupLoads = kSupPayLoads + kSupScLoads;

// One slice of a lane's operand data: payload words (groups 0..3 = A rows
// 32i + l%32 of the wave's 128, groups 4..7 = B rows 32j + l%32; word kk =
// k-step kk) and per group the row's scale word, replaced at k-step 0 by the
// two block scales of the lane's half as fp16 bit patterns (low half:
// k-steps 0, 1; high half: k-steps 2, 3).
struct RegSlice {
    uint32_t w[8][4];
    uint32_t s[8];
};

__device__ __forceinline__ uint32_t half_scales(uint32_t word, uint32_t sel) {
    return __builtin_amdgcn_perm(0u, word, sel) << 7;
}

// Slice SL of the stage (P, S) into R.  pa / pb: byte offsets of the lane's
// first A / B stage row (group 0); xo: the lane's chunk offset for this slice.
template <int SL>
__device__ __forceinline__ void read_sup_slice(RegSlice& R, const uint8_t* P, const uint8_t* S,
                                               int pa, int pb, int xo) {
#pragma unroll
    for (int g = 0; g < 8; ++g) {
        const int row_off = (g < 4 ? pa : pb) + (g & 3) * 32 * kSupRowBytes;
        const uint4 v = *reinterpret_cast<const uint4*>(P + row_off + xo);
        R.w[g][0] = v.x; R.w[g][1] = v.y; R.w[g][2] = v.z; R.w[g][3] = v.w;
    }
#pragma unroll
    for (int g = 0; g < 8; ++g) {
        const int srow_off = ((g < 4 ? pa : pb) / kSupRowBytes + (g & 3) * 32) * (kSupK * 4);
        R.s[g] = *reinterpret_cast<const uint32_t*>(S + srow_off + SL * 4);
    }
}

template <int HSEL>
__device__ __forceinline__ f16x8_t decode_frag(uint32_t w, uint32_t s2) {
    const f16x2_t sp = __builtin_bit_cast(f16x2_t, s2);
    const f16x2_t sc = __builtin_shufflevector(sp, sp, HSEL, HSEL);   // op_sel picks the half
    const f16x2_t v0 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 0.125f, 0) * sc;
    const f16x2_t v1 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 0.125f, 1) * sc;
    const f16x2_t v2 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 0.125f, 2) * sc;
    const f16x2_t v3 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 0.125f, 3) * sc;
    return f16x8_t{v0[0], v0[1], v1[0], v1[1], v2[0], v2[1], v3[0], v3[1]};
}

// k-step KK of a slice into MFMA fragments.  At KK = 0 the raw scale words
// read from LDS are first turned into the lane half's two fp16 scales (done
// here, a k-step after the LDS reads were issued, so that no wait for them
// lands among the matrix-core instructions).
template <int KK>
__device__ __forceinline__ void decode_kstep(Frags& f, RegSlice& R, uint32_t sel) {
    if (KK == 0) {
#pragma unroll
        for (int g = 0; g < 8; ++g) {
            R.s[g] = half_scales(R.s[g], sel);
            // opaque to the compiler, which would otherwise rebuild the high
            // half with a shift instead of selecting it by op_sel
            asm("" : "+v"(R.s[g]));
        }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) f.a[i] = decode_frag<KK / 2>(R.w[i][KK], R.s[i]);
#pragma unroll
    for (int j = 0; j < 4; ++j) f.b[j] = decode_frag<KK / 2>(R.w[4 + j][KK], R.s[4 + j]);
}

// Direct global->LDS loads written as instructions the compiler does not
// model: it would otherwise wait for every outstanding direct load before any
// LDS read (it cannot tell the stage arrays apart), which would remove the
// overlap.  The kernel counts them itself with vmcnt.  The LDS destination of
// lane l is m0 + 16 l.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
    return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lds_void_ptr)p);
}

// Calls f(integral_constant<int, i>) for i in [I0, I1).
template <int I0, int I1, typename F>
__device__ __forceinline__ void static_for(F&& f) {
    if constexpr (I0 < I1) {
        f(std::integral_constant<int, I0>{});
        static_for<I0 + 1, I1>(f);
    }
}

// Buffer resource of a raw byte range [base, base + bytes): loads whose
// per-lane offset falls outside it are dropped by the hardware.
typedef int i32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ i32x4_t buffer_rsrc(const void* base, uint32_t bytes) {
    const uint64_t a = (uint64_t)(uintptr_t)base;
    i32x4_t r;
    r[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
    r[1] = __builtin_amdgcn_readfirstlane((int)(uint32_t)(a >> 32));   // stride 0
    r[2] = (int)bytes;
    r[3] = 0x00020000;                                                   // 32-bit data format
    return r;
}

// 16 bytes per lane from rsrc at voff + soff into LDS at lds + OFF + 16 lane
// (the LDS offset is added inside the instruction sequence so that the
// compiler does not keep one register per destination).
template <int OFF>
__device__ __forceinline__ void dma_buf_x4(i32x4_t rsrc, uint32_t voff, uint32_t soff, uint32_t lds) {
    asm volatile("s_add_u32 m0, %3, %4\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, %2 offen lds"
                 :: "v"(voff), "s"(rsrc), "s"(soff), "s"(lds), "i"(OFF) : "memory", "m0", "scc");
}

// vmcnt(n) with expcnt and lgkmcnt left at their maxima (n < 64).
template <int n>
__device__ __forceinline__ void wait_vmem() {
    static_assert(n >= 0 && n < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((n & 15) | ((n >> 4) << 14) | 0x0F70);
}

// Per-lane source of a wave's stage loads for one output tile: byte offsets
// of the lane's first payload chunk and of its two scale rows.
struct SupSrc {
    uint32_t off0, so0, so1;
};

// A wave's share of the loads of one stage: payload loads i in [I0, I1)
// (1 KB each: 8 stage rows of 128 B, lane l -> row 8i + l/8 of the wave's
// 128, position l % 8) and, with SC, its two scale loads (64 rows x 16 B).
// Payload rows past the matrix fall outside the buffer and are dropped (they
// only feed discarded outputs); scale rows are clamped when the tile is set up.
struct SupLoader {
    i32x4_t pay, sca;        // payload and scale buffers of this wave's matrix (A or B)
    uint32_t rows8;          // bytes of 8 payload rows
    uint32_t ldp, lds;       // this wave's LDS offsets inside a payload / scale stage

    template <int I0, int I1, bool SC>
    __device__ __forceinline__ void issue(uint32_t P, uint32_t S, const SupSrc& src, int64_t G) const {
        const uint32_t gp = (uint32_t)G * kSupRowBytes;
        const uint32_t pl = P + ldp;
        static_for<I0, I1>([&](auto ic) {
            constexpr int i = decltype(ic)::value;
            dma_buf_x4<i * 1024>(pay, src.off0 + i * rows8, gp, pl);
        });
        if (SC) {
            const uint32_t gs = (uint32_t)G * 16;
            const uint32_t sl = S + lds;
            dma_buf_x4<0>(sca, src.so0, gs, sl);
            dma_buf_x4<1024>(sca, src.so1, gs, sl);
        }
    }
};

// Split of the last, partial wave of tiles: with T tiles on P CUs, the first
// Tdp = T - r tiles (whole waves) are whole work items; each of the r
// leftover tiles becomes `parts` items over equal ranges of its stages, which
// write fp32 partial tiles; a second kernel adds each tile's partials in part
// order (so the sum is deterministic) and stores it.
struct SplitPlan {
    int Tdp;                 // whole-tile items
    int parts;               // items per leftover tile (1: no split)
    float* part;             // [r][parts][4 waves][16 acc (i, j)][4 runs][64 lanes][4] fp32 partials
};

// Origin of logical tile t: workgroups are dispatched round-robin over the
// XCDs, so logical tiles are remapped to give each XCD a contiguous range,
// walked in groups of kGroupM tile rows (column-major inside a group) so
// that tiles running together on one XCD share A and B rows in its L2.
__device__ __forceinline__ void tile_origin(int t, int tiles_m, int tiles_n, int64_t& m0, int64_t& n0) {
    const int ntiles = tiles_m * tiles_n;
    if (ntiles % kXcds == 0) t = (t % kXcds) * (ntiles / kXcds) + t / kXcds;
    const int group_tiles = kGroupM * tiles_n;
    const int g = t / group_tiles;
    const int first_m = g * kGroupM;
    const int gm = min(tiles_m - first_m, kGroupM);
    const int rr = t - g * group_tiles;
    m0 = (int64_t)(first_m + rr % gm) * BM;
    n0 = (int64_t)(rr / gm) * BN;
}

constexpr bool kStaggerSplit = true;

// One work item: a whole tile (split_j < 0) or part `part` of leftover tile
// split_j, over stages [g0, g1).  With an even stage count per tile, part
// boundaries fall on even stages so every item has an even length.
struct WorkItem {
    int t, split_j, part, g0, g1;
};

__device__ __forceinline__ WorkItem work_item(int it, const SplitPlan& sp, int NG) {
    WorkItem w;
    if (it < sp.Tdp) {
        w.t = it; w.split_j = -1; w.part = 0; w.g0 = 0; w.g1 = NG;
        return w;
    }
    const int s = it - sp.Tdp;
    w.split_j = s / sp.parts;
    w.part = s - w.split_j * sp.parts;
    w.t = sp.Tdp + w.split_j;
    const int unit = (NG % 2 == 0) ? 2 : 1;
    const int nu = NG / unit;
    w.g0 = unit * ((nu * w.part) / sp.parts);
    w.g1 = unit * ((nu * (w.part + 1)) / sp.parts);
    return w;
}

// LDS bytes per wave for the epilogue's row transposition (32 rows x 128 B).
constexpr int kEpiBytes = 4096;

// Orders a wave's LDS writes before its own later LDS reads of what other
// lanes wrote (and those reads before the next writes): the LDS serves one
// wave's instructions in order, so the compiler only must not move memory
// accesses across this point and the data must have landed.
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_s_waitcnt(0xC07F);              // lgkmcnt(0)
    asm volatile("" ::: "memory");
}


// Epilogue of one work item.  Element e of accumulator (i, j) is row
// 32i + l%32, column 32j + 8(e/4) + 4(l/32) + e%4 of the wave's 128 x 128
// block (the products are issued as B x A^T).  A split part stores its fp32
// partial; a whole tile stores alpha * value through a buffer resource over
// C, where an out-of-range offset drops the store, which masks rows and
// columns past C without branches.  VEC (a launch-time choice,
// vector_epilogue): N % 8 == 0 for bf16, N % 4 == 0 for fp32, where every
// run of 8 (4) output columns lies wholly inside C or wholly past it;
// otherwise each element is masked on its own.  With VEC the values pass through the wave's 4 KB of LDS
// (`ep`), 32 rows x 128 bytes at a time, and leave as stores of 128
// contiguous bytes per row (8 rows per instruction): a lane holds one row,
// so storing straight from the accumulators writes 32 rows x 32 bytes per
// instruction, which the memory path serves at a quarter of the rate.  In
// the staging area the 16-byte chunk c of row x sits at c ^ ((x / 2) % 8),
// which spreads both the writes and the reads over all LDS banks.
template <bool OUT_BF16, bool VEC>
__device__ __forceinline__ void store_item(f32x16_t (&acc)[4][4], const WorkItem& cur,
                                           const SplitPlan& sp, int M, int N, int tiles_m, int tiles_n,
                                           int wave, int lane, float alpha, void* __restrict__ C,
                                           uint8_t* __restrict__ ep) {
    const int wm = wave >> 1, wn = wave & 1;
    const int r = lane & 31, hi = lane >> 5;
    if (cur.split_j >= 0) {
        // one part of a leftover tile: fp32 partial, [acc (i, j)][run g]
        // [lane][4] so that every store is 16 bytes per lane, 1 KB per wave
        const __amdgpu_buffer_rsrc_t pr = __builtin_amdgcn_make_buffer_rsrc(
            sp.part + ((int64_t)cur.split_j * sp.parts + cur.part) * 65536, 0, 65536 * 4, 0x00020000);
        const uint32_t vo = (uint32_t)(wave * 65536 + lane * 16);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const f32x4_t v = {acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2],
                                       acc[i][j][4 * g + 3]};
                    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, v), pr, vo,
                                                           ((i * 4 + j) * 4 + g) * 1024, 0);
                }
            __builtin_amdgcn_sched_barrier(0);
        }
        return;
    }
    constexpr uint32_t esz = OUT_BF16 ? 2 : 4;
    constexpr uint32_t kOff = 0x80000000u;               // past every buffer
    const __amdgpu_buffer_rsrc_t cr =
        __builtin_amdgcn_make_buffer_rsrc(C, 0, (int)((uint32_t)M * (uint32_t)N * esz), 0x00020000);
    int64_t m0, n0;
    tile_origin(cur.t, tiles_m, tiles_n, m0, n0);
    const int mrow = (int)m0 + wm * 128 + r;
    if (VEC) {
        // Write side: lane (r, hi) puts its row's values of the current
        // 32-row block; read side: lane l takes chunk l % 8 of row
        // l / 8 + 8t.  bf16: a store's row lies past C exactly when its
        // offset does (the column run is checked once), so the per-store
        // offset is the lane's base plus a uniform row offset.  The sum is
        // formed in the vector offset, so that the range check sees the
        // whole offset (the compiler's buffer intrinsics document the scalar
        // offset as outside that check) and stays below 2^32 by the launch
        // condition.
        const int wsw = (r >> 1) & 7;
        const int rr = lane >> 3, rc = lane & 7;
        const uint32_t mb = (uint32_t)((int)m0 + wm * 128 + rr);
        uint8_t* const wrow = ep + r * 128;
        const uint8_t* rd[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) rd[t] = ep + (rr + 8 * t) * 128 + ((rc ^ (((rr + 8 * t) >> 1) & 7)) << 4);
        if (OUT_BF16) {
            // round q = 2i + h: 32 rows x 64 columns (j = 2h, 2h + 1)
            uint32_t vb[2];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int n = (int)n0 + wn * 128 + 64 * h + 8 * rc;
                vb[h] = n < N ? (mb * (uint32_t)N + (uint32_t)n) * 2u : kOff;
            }
            auto pack = [&](int q, u32x2_t (&v)[8]) {
                const int i = q >> 1, h = q & 1;
#pragma unroll
                for (int jj = 0; jj < 2; ++jj)
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        const f32x16_t& a = acc[i][2 * h + jj];
                        v[4 * jj + g] = u32x2_t{pack_bf16x2(alpha * a[4 * g], alpha * a[4 * g + 1]),
                                                pack_bf16x2(alpha * a[4 * g + 2], alpha * a[4 * g + 3])};
                    }
            };
            // the round's accumulators are read only where they are packed:
            // an empty statement that takes them as VGPR operands is where
            // the compiler copies each one out of the AccVGPRs, once (with
            // AccVGPR operands it moved them to other AccVGPRs first, 32
            // moves per round)
            auto take = [&](int q, u32x2_t (&v)[8]) {
                asm volatile("" : "+v"(acc[q >> 1][2 * (q & 1)]), "+v"(acc[q >> 1][2 * (q & 1) + 1]));
                pack(q, v);
            };
            u32x2_t v[8], vn[8];
            take(0, v);
#pragma unroll
            for (int q = 0; q < 8; ++q) {
#pragma unroll
                for (int jj = 0; jj < 2; ++jj)
#pragma unroll
                    for (int g = 0; g < 4; ++g)
                        *reinterpret_cast<u32x2_t*>(wrow + (((4 * jj + g) ^ wsw) << 4) + hi * 8) = v[4 * jj + g];
                // the next round's values are formed while these writes land
                if (q < 7) take(q + 1, vn);
                wave_lds_sync();
                const int i = q >> 1, h = q & 1;
                // all four reads first: the compiler cannot tell that the
                // buffer stores do not alias the LDS, so a read written
                // after a store would wait for it (one LDS round trip per
                // store instead of one per round)
                u32x4_t d[4];
#pragma unroll
                for (int t = 0; t < 4; ++t) d[t] = *reinterpret_cast<const u32x4_t*>(rd[t]);
#pragma unroll
                for (int t = 0; t < 4; ++t)
                    __builtin_amdgcn_raw_buffer_store_b128(d[t], cr, vb[h] + (uint32_t)((32 * i + 8 * t) * N * 2),
                                                           0, 0);
                wave_lds_sync();
                if (q < 7) {
#pragma unroll
                    for (int k = 0; k < 8; ++k) v[k] = vn[k];
                }
            }
        } else {
            // round q = 4i + j: 32 rows x 32 columns; the next round's
            // values are formed while a round's writes land
            auto take = [&](int q, f32x4_t (&v)[4]) {
                const int i = q >> 2, j = q & 3;
                asm volatile("" : "+v"(acc[i][j]));      // read out here, once
#pragma unroll
                for (int g = 0; g < 4; ++g)
                    v[g] = f32x4_t{alpha * acc[i][j][4 * g], alpha * acc[i][j][4 * g + 1],
                                   alpha * acc[i][j][4 * g + 2], alpha * acc[i][j][4 * g + 3]};
            };
            f32x4_t v[4], vn[4];
            take(0, v);
#pragma unroll
            for (int q = 0; q < 16; ++q) {
                const int i = q >> 2, j = q & 3;
#pragma unroll
                for (int g = 0; g < 4; ++g) *reinterpret_cast<f32x4_t*>(wrow + (((2 * g + hi) ^ wsw) << 4)) = v[g];
                if (q < 15) take(q + 1, vn);
                wave_lds_sync();
                u32x4_t d[4];                               // all reads before the stores
#pragma unroll
                for (int t = 0; t < 4; ++t) d[t] = *reinterpret_cast<const u32x4_t*>(rd[t]);
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    const int m = (int)mb + 32 * i + 8 * t;
                    const int n = (int)n0 + wn * 128 + 32 * j + 4 * rc;
                    const uint32_t vo = (m < M && n < N) ? ((uint32_t)m * (uint32_t)N + (uint32_t)n) * 4u : kOff;
                    __builtin_amdgcn_raw_buffer_store_b128(d[t], cr, vo, 0, 0);
                }
                wave_lds_sync();
                if (q < 15) {
#pragma unroll
                    for (int g = 0; g < 4; ++g) v[g] = vn[g];
                }
            }
        }
        return;
    }
    const int ncol = (int)n0 + wn * 128 + hi * 4;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int m = mrow + 32 * i;
        const uint32_t rbase = ((uint32_t)m * (uint32_t)N + (uint32_t)ncol) * esz;
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int n = ncol + 32 * j + 8 * g;
                const float v0 = alpha * acc[i][j][4 * g + 0], v1 = alpha * acc[i][j][4 * g + 1];
                const float v2 = alpha * acc[i][j][4 * g + 2], v3 = alpha * acc[i][j][4 * g + 3];
                const uint32_t imm = (uint32_t)(32 * j + 8 * g) * esz;
                const float vv[4] = {v0, v1, v2, v3};
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const uint32_t vo = (m < M && n + q < N) ? rbase : kOff;
                    if (OUT_BF16) {
                        __builtin_amdgcn_raw_buffer_store_b16(
                            (unsigned short)pack_bf16x2(vv[q], 0.0f), cr, vo + imm + q * esz, 0, 0);
                    } else {
                        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(vv[q]), cr,
                                                              vo + imm + q * esz, 0, 0);
                    }
                }
            }
        __builtin_amdgcn_sched_barrier(0);
    }
}

// Register-decode GEMM, persistent: workgroup w runs items w, w + grid, ...
// (whole tiles first, then split parts).  During the last two stages of an
// item the next item's first two stages are loaded, so its epilogue and the
// next item's start overlap those loads instead of waiting for them.  Items
// must have an even number of stages when a workgroup runs more than one
// (the stage buffers alternate and every item starts in buffer 0).  Sizes:
// every operand, C and the partial workspace span less than 2^31 bytes.
template <int BMODE, bool OUT_BF16, bool VEC>
__global__ __launch_bounds__(kGemmThreads, 1) void gemm_fp4_reg_kernel(
    int M, int N, int K, int tiles_m, int tiles_n, int items, SplitPlan sp,
    const uint8_t* __restrict__ A, const uint8_t* __restrict__ As, const float* __restrict__ a_dec,
    const uint8_t* __restrict__ B, const uint8_t* __restrict__ Bs, const float* __restrict__ b_dec,
    void* __restrict__ C, float amul) {
    __shared__ __attribute__((aligned(16))) uint8_t sP0[kSupPayload];
    __shared__ __attribute__((aligned(16))) uint8_t sP1[kSupPayload];
    __shared__ __attribute__((aligned(16))) uint8_t sC0[kSupScales];
    __shared__ __attribute__((aligned(16))) uint8_t sC1[kSupScales];
    __shared__ __attribute__((aligned(16))) uint8_t sE[kGemmThreads / 64 * kEpiBytes];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1, wn = wave & 1;
    const int r = lane & 31, hi = lane >> 5;

    const int kbt = K / 16;                          // scale bytes per row
    const int NG = K / (kSupK * BK);                 // stages of a whole tile

    // Loads: waves 0, 1 bring A stage rows 0..255, waves 2, 3 B rows 256..511.
    const bool isA = wave < 2;
    const int xw = 128 * (wave & 1);                 // first stage row of the wave within A or B
    const int brows = BMODE == (int)BScale::Row ? N : (N + 15) / 16;   // rows of the B scale matrix
    SupLoader L;
    L.pay = isA ? buffer_rsrc(A, (uint32_t)M * kbt * 8) : buffer_rsrc(B, (uint32_t)N * kbt * 8);
    L.sca = isA ? buffer_rsrc(As, (uint32_t)M * kbt) : buffer_rsrc(Bs, (uint32_t)brows * kbt);
    L.rows8 = (uint32_t)(64 * kbt);
    L.ldp = (uint32_t)(128 * wave * kSupRowBytes);
    L.lds = (uint32_t)(128 * wave * kSupK * 4);
    const uint32_t chunk16 = (uint32_t)(((lane & 7) ^ ((lane >> 3) & 7)) * 16);
    auto src_of = [&](int t) {
        int64_t m0, n0;
        tile_origin(t, tiles_m, tiles_n, m0, n0);
        const int x0 = (int)(isA ? m0 : n0) + xw;
        SupSrc q;
        q.off0 = (uint32_t)(x0 + (lane >> 3)) * (uint32_t)(kbt * 8) + chunk16;
        const int xa = x0 + lane, xb = x0 + 64 + lane;
        if (isA) {
            q.so0 = (uint32_t)min(xa, M - 1) * kbt;
            q.so1 = (uint32_t)min(xb, M - 1) * kbt;
        } else {
            const int na = min(xa, N - 1), nb = min(xb, N - 1);
            q.so0 = (uint32_t)(BMODE == (int)BScale::Row ? na : (na >> 4)) * kbt;
            q.so1 = (uint32_t)(BMODE == (int)BScale::Row ? nb : (nb >> 4)) * kbt;
        }
        return q;
    };
    const uint32_t P0 = lds_addr(sP0), P1 = lds_addr(sP1), S0 = lds_addr(sC0), S1 = lds_addr(sC1);

    // Read offsets of the lane: first A / B stage rows and per-slice chunk.
    const int pa = (wm * 128 + r) * kSupRowBytes;
    const int pb = (BM + wn * 128 + r) * kSupRowBytes;
    const int x0 = ((0 + hi) ^ (r & 7)) * 16, x1 = ((2 + hi) ^ (r & 7)) * 16;
    const int x2 = ((4 + hi) ^ (r & 7)) * 16, x3 = ((6 + hi) ^ (r & 7)) * 16;
    const uint32_t sel = hi ? 0x0C030C02u : 0x0C010C00u;

    f32x16_t acc[4][4];
    RegSlice R0, R1;
    Frags F0, F1;

    // Items of this workgroup: w, w + grid, ...  Odd workgroups whose last
    // item is a split part run that part first, so that their tile
    // boundaries fall between those of the even ones and the output stores
    // of all CUs do not come in one burst.
    const int grid = (int)gridDim.x;
    const int nw = (items - (int)blockIdx.x + grid - 1) / grid;
    const int last_it = (int)blockIdx.x + (nw - 1) * grid;
    const bool rot = kStaggerSplit && (blockIdx.x & 1) && nw > 1 && last_it >= sp.Tdp;
    auto item_at = [&](int k) {
        return rot ? (k == 0 ? last_it : (int)blockIdx.x + (k - 1) * grid) : (int)blockIdx.x + k * grid;
    };

    // prologue: stages 0 and 1 of the first item in flight, stage 0 complete
    // everywhere
    {
        const WorkItem w = work_item(item_at(0), sp, NG);
        const SupSrc q = src_of(w.t);
        L.issue<0, kSupPayLoads, true>(P0, S0, q, w.g0);
        L.issue<0, kSupPayLoads, true>(P1, S1, q, min(w.g0 + 1, w.g1 - 1));
        wait_vmem<kSupLoads>();
        __syncthreads();
    }

    // Only the item position is carried from one item to the next; everything
    // else is rebuilt from it, which keeps the registers free for the
    // epilogue.  The item's first stage is in buffer 0 and complete.
    for (int k = 0;; ++k) {
        const int it = item_at(k);
        const WorkItem cur = work_item(it, sp, NG);
        const SupSrc scur = src_of(cur.t);
        const bool has_next = k + 1 < nw;
        const WorkItem nxt = work_item(has_next ? item_at(k + 1) : it, sp, NG);
        const SupSrc snxt = src_of(nxt.t);
        read_sup_slice<0>(R0, sP0, sC0, pa, pb, x0);
        decode_kstep<0>(F0, R0, sel);
        // stage index of the load sequence -> (source, stage): this item's,
        // the next item's first stages, or (no next item) this item's last
        // again; chosen by selects so that the stage code stays branch-free
        const int gshift = has_next ? nxt.g0 - cur.g1 : -1;
        const int gclamp = has_next ? 0x7FFFFFFF : cur.g1 - 1;

        auto issue_for = [&](auto I0c, auto I1c, auto SCc, uint32_t ldP, uint32_t ldS, int Gt) {
            constexpr int I0v = decltype(I0c)::value, I1v = decltype(I1c)::value;
            constexpr bool SCv = decltype(SCc)::value;
            const bool in_cur = Gt < cur.g1;
            const int Gl = in_cur ? Gt : min(Gt + gshift, gclamp);
            SupSrc q;
            q.off0 = in_cur ? scur.off0 : snxt.off0;
            q.so0 = in_cur ? scur.so0 : snxt.so0;
            q.so1 = in_cur ? scur.so1 : snxt.so1;
            L.issue<I0v, I1v, SCv>(ldP, ldS, q, Gl);
        };

#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
#pragma unroll
                for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;
                asm volatile("" : "+a"(acc[i][j]));      // zeros go straight to the AccVGPRs
            }

        // One slice.  Slices 0..2 of a stage read the next slice of the same
        // stage; slice 3 first waits for the next stage (loaded during the
        // previous stage), synchronizes, starts the loads of stage G+2 into
        // the buffer just consumed, and reads slice 0 of the next stage.
        // A k-step's decode is about 76 VALU instructions against its 16
        // MFMAs, so each MFMA is followed by up to five of them (with four
        // the remainder bunches up behind the last MFMA; measured per GEMM:
        // five slots 0.4-1.1% faster than four, three or eight 2-4% slower).
        auto slice = [&](auto SLc, int G, const uint8_t* Pc, const uint8_t* Sc, const uint8_t* Pn,
                         const uint8_t* Sn, uint32_t ldP, uint32_t ldS, RegSlice& Rc, RegSlice& Rn) {
            constexpr int SL = decltype(SLc)::value;
            using Z = std::integral_constant<int, 0>;
            using C6 = std::integral_constant<int, 6>;
            using C12 = std::integral_constant<int, 12>;
            using CP = std::integral_constant<int, kSupPayLoads>;
            using F = std::integral_constant<bool, false>;
            using T = std::integral_constant<bool, true>;
            decode_kstep<1>(F1, Rc, sel);
            mfma16_t(acc, F0);
            kstep_schedule<0, 0, 5>();
            __builtin_amdgcn_sched_barrier(0);
            if (SL == 3) {
                wait_vmem<0>();
                __syncthreads();
                read_sup_slice<0>(Rn, Pn, Sn, pa, pb, x0);
                issue_for(Z{}, C6{}, F{}, ldP, ldS, G + 2);
            } else {
                read_sup_slice<SL + 1>(Rn, Pc, Sc, pa, pb, SL == 0 ? x1 : (SL == 1 ? x2 : x3));
            }
            decode_kstep<2>(F0, Rc, sel);
            mfma16_t(acc, F1);
            kstep_schedule<16, 0, 5>();
            __builtin_amdgcn_sched_barrier(0);
            if (SL == 3) issue_for(C6{}, C12{}, F{}, ldP, ldS, G + 2);
            decode_kstep<3>(F1, Rc, sel);
            mfma16_t(acc, F0);
            kstep_schedule<0, 0, 5>();
            __builtin_amdgcn_sched_barrier(0);
            if (SL == 3) issue_for(C12{}, CP{}, T{}, ldP, ldS, G + 2);
            decode_kstep<0>(F0, Rn, sel);
            mfma16_t(acc, F1);
            kstep_schedule<0, 0, 5>();
            __builtin_amdgcn_sched_barrier(0);
        };
        using I0 = std::integral_constant<int, 0>;
        using I1 = std::integral_constant<int, 1>;
        using I2 = std::integral_constant<int, 2>;
        using I3 = std::integral_constant<int, 3>;
        auto stage = [&](int G, const uint8_t* Pc, const uint8_t* Sc, const uint8_t* Pn,
                         const uint8_t* Sn, uint32_t ldP, uint32_t ldS) {
            slice(I0{}, G, Pc, Sc, Pn, Sn, ldP, ldS, R0, R1);
            slice(I1{}, G, Pc, Sc, Pn, Sn, ldP, ldS, R1, R0);
            slice(I2{}, G, Pc, Sc, Pn, Sn, ldP, ldS, R0, R1);
            slice(I3{}, G, Pc, Sc, Pn, Sn, ldP, ldS, R1, R0);
        };
        int G = cur.g0;
        for (; G + 1 < cur.g1; G += 2) {
            stage(G, sP0, sC0, sP1, sC1, P0, S0);
            stage(G + 1, sP1, sC1, sP0, sC0, P1, S1);
        }
        if (G < cur.g1) stage(G, sP0, sC0, sP1, sC1, P0, S0);   // odd stage count (single item)

        store_item<OUT_BF16, VEC>(acc, cur, sp, M, N, tiles_m, tiles_n, wave, lane,
                                  (a_dec[0] * b_dec[0]) * amul, C, sE + wave * kEpiBytes);   // operands were scaled by 2^-3
        if (!has_next) break;
    }
    wait_vmem<0>();                                  // no load outlives the kernel's LDS
}

// ===================================================================== //
// E8M0 blocks of 32 (MXFP4 arrangement): the gfx950 scaled FP4 matrix    //
// instruction multiplies E2M1 payloads and applies the per-32 power-of-  //
// two scales itself, so nothing is decoded.                              //
// ===================================================================== //
// v_mfma_scale_f32_32x32x64_f8f6f4 with both formats E2M1: lane l supplies
// row l%32 and k = 32(l/32) .. +31 as 16 payload bytes (the stored order),
// plus the E8M0 byte of that row and k-half; the product of the two scale
// powers is exact and the accumulation is binary32.  Same tiles, stages,
// persistent items and epilogue as the register-decode kernel; a stage row
// holds 128 payload bytes and 8 scale bytes (256 k).
constexpr int kMxScaleStage = kSupRows * 8;               // 4 KB of scales per stage
constexpr int kMxScLoads = 4;                             // 4 x 256 B per wave
constexpr int kMxLoads = kSupPayLoads + kMxScLoads;

// 4 bytes per lane from rsrc at voff + soff into LDS at lds + OFF + 4 lane.
template <int OFF>
__device__ __forceinline__ void dma_buf_x1(i32x4_t rsrc, uint32_t voff, uint32_t soff, uint32_t lds) {
    asm volatile("s_add_u32 m0, %3, %4\n\ts_nop 0\n\tbuffer_load_dword %0, %1, %2 offen lds"
                 :: "v"(voff), "s"(rsrc), "s"(soff), "s"(lds), "i"(OFF) : "memory", "m0", "scc");
}

// Per-lane load sources of one tile: first payload chunk; the scale bytes
// of rows x0 + 32u + l/2 (dword l%2 of their 8 stage bytes), u = 0..3.
struct MxSrc {
    uint32_t off0;
    uint32_t so[4];
};

struct MxLoader {
    i32x4_t pay, sca;
    uint32_t rows8;          // bytes of 8 payload rows
    uint32_t ldp, lds;       // this wave's LDS offsets inside a payload / scale stage

    template <int I0, int I1, bool SC>
    __device__ __forceinline__ void issue(uint32_t P, uint32_t S, const MxSrc& src, int G) const {
        const uint32_t gp = (uint32_t)G * kSupRowBytes;
        const uint32_t pl = P + ldp;
        static_for<I0, I1>([&](auto ic) {
            constexpr int i = decltype(ic)::value;
            dma_buf_x4<i * 1024>(pay, src.off0 + i * rows8, gp, pl);
        });
        if (SC) {
            const uint32_t gs = (uint32_t)G * 8;
            const uint32_t sl = S + lds;
            dma_buf_x1<0>(sca, src.so[0], gs, sl);
            dma_buf_x1<256>(sca, src.so[1], gs, sl);
            dma_buf_x1<512>(sca, src.so[2], gs, sl);
            dma_buf_x1<768>(sca, src.so[3], gs, sl);
        }
    }
};

// One slice of a lane's operands: 16 payload bytes of each of its 4 A and 4
// B rows (groups 0..3 = A rows 32i + l%32, 4..7 = B rows 32j + l%32).
struct MxSlice {
    uint32_t w[8][4];
};

template <int SL>
__device__ __forceinline__ void read_mx_slice(MxSlice& R, const uint8_t* P, int pa, int pb, int xo) {
#pragma unroll
    for (int g = 0; g < 8; ++g) {
        const int row_off = (g < 4 ? pa : pb) + (g & 3) * 32 * kSupRowBytes;
        const uint4 v = *reinterpret_cast<const uint4*>(P + row_off + xo);
        R.w[g][0] = v.x; R.w[g][1] = v.y; R.w[g][2] = v.z; R.w[g][3] = v.w;
    }
}

// The 8 scale bytes (256 k) of each of the lane's 8 rows, shifted right by
// one byte in the upper lane half so that, for slice SL, the lane's byte
// (2 SL + l/32) sits at byte 2 (SL % 2) of dword SL / 2.
__device__ __forceinline__ void read_mx_scales(uint32_t (&sc)[8][2], const uint8_t* S, int ra, int rb,
                                               int hi) {
#pragma unroll
    for (int g = 0; g < 8; ++g) {
        const int row = (g < 4 ? ra : rb) + (g & 3) * 32;
        const uint2 v = *reinterpret_cast<const uint2*>(S + row * 8);
        sc[g][0] = v.x >> (8 * hi);
        sc[g][1] = v.y >> (8 * hi);
    }
}

// One scaled FP4 product accumulated in place.  Written as an instruction
// with a read-write accumulator operand: the compiler's builtin for it has no
// accumulate-in-place form, and its register allocator then moves every
// accumulator through a temporary around each product.  SEL picks byte SEL
// of both scale registers.
typedef int i32x4v_t __attribute__((ext_vector_type(4)));
template <int SEL>
__device__ __forceinline__ void mfma_mx(f32x16_t& acc, const i32x4v_t& a, const i32x4v_t& b, uint32_t sa,
                                        uint32_t sb) {
    static_assert(SEL == 0 || SEL == 2, "scale byte 0 or 2");
    // volatile: kept in program order with the waits placed after them
    if (SEL == 0)
        asm volatile("v_mfma_scale_f32_32x32x64_f8f6f4 %0, %1, %2, %0, %3, %4 op_sel_hi:[0,0,0] cbsz:4 blgp:4"
                     : "+a"(acc) : "v"(a), "v"(b), "v"(sa), "v"(sb));
    else
        asm volatile("v_mfma_scale_f32_32x32x64_f8f6f4 %0, %1, %2, %0, %3, %4 op_sel_hi:[1,1,0] cbsz:4 blgp:4"
                     : "+a"(acc) : "v"(a), "v"(b), "v"(sa), "v"(sb));
}

template <int SL>
__device__ __forceinline__ void mfma_mx16(f32x16_t (&acc)[4][4], const MxSlice& R, const uint32_t (&sc)[8][2]) {
    constexpr int d = SL / 2, sel = 2 * (SL % 2);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const i32x4v_t a = {(int)R.w[4 + j][0], (int)R.w[4 + j][1], (int)R.w[4 + j][2], (int)R.w[4 + j][3]};
            const i32x4v_t b = {(int)R.w[i][0], (int)R.w[i][1], (int)R.w[i][2], (int)R.w[i][3]};
            // products issued as B x A^T (see store_item)
            mfma_mx<sel>(acc[i][j], a, b, sc[4 + j][d], sc[i][d]);
        }
}

template <bool OUT_BF16, bool VEC>
__global__ __launch_bounds__(kGemmThreads, 1) void gemm_mx_kernel(
    int M, int N, int K, int tiles_m, int tiles_n, int items, SplitPlan sp,
    const uint8_t* __restrict__ A, const uint8_t* __restrict__ As, const float* __restrict__ a_dec,
    const uint8_t* __restrict__ B, const uint8_t* __restrict__ Bs, const float* __restrict__ b_dec,
    void* __restrict__ C) {
    __shared__ __attribute__((aligned(16))) uint8_t sP0[kSupPayload];
    __shared__ __attribute__((aligned(16))) uint8_t sP1[kSupPayload];
    __shared__ __attribute__((aligned(16))) uint8_t sC0[kMxScaleStage];
    __shared__ __attribute__((aligned(16))) uint8_t sC1[kMxScaleStage];
    __shared__ __attribute__((aligned(16))) uint8_t sE[kGemmThreads / 64 * kEpiBytes];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1, wn = wave & 1;
    const int r = lane & 31, hi = lane >> 5;

    const int kb32 = K / 32;                         // scale bytes per row
    const int NG = K / (kSupK * BK);                 // stages of a whole tile

    // Loads: waves 0, 1 bring A stage rows 0..255, waves 2, 3 B rows 256..511.
    const bool isA = wave < 2;
    const int xw = 128 * (wave & 1);
    MxLoader L;
    L.pay = isA ? buffer_rsrc(A, (uint32_t)M * (uint32_t)(K / 2)) : buffer_rsrc(B, (uint32_t)N * (uint32_t)(K / 2));
    L.sca = isA ? buffer_rsrc(As, (uint32_t)M * kb32) : buffer_rsrc(Bs, (uint32_t)N * kb32);
    L.rows8 = (uint32_t)(8 * (K / 2));
    L.ldp = (uint32_t)(128 * wave * kSupRowBytes);
    L.lds = (uint32_t)(128 * wave * 8);
    const uint32_t chunk16 = (uint32_t)(((lane & 7) ^ ((lane >> 3) & 7)) * 16);
    const int rmax = (isA ? M : N) - 1;
    auto src_of = [&](int t) {
        int64_t m0, n0;
        tile_origin(t, tiles_m, tiles_n, m0, n0);
        const int x0 = (int)(isA ? m0 : n0) + xw;
        MxSrc q;
        q.off0 = (uint32_t)(x0 + (lane >> 3)) * (uint32_t)(K / 2) + chunk16;
#pragma unroll
        for (int u = 0; u < 4; ++u)
            q.so[u] = (uint32_t)min(x0 + 32 * u + (lane >> 1), rmax) * (uint32_t)kb32 + 4u * (lane & 1);
        return q;
    };
    const uint32_t P0 = lds_addr(sP0), P1 = lds_addr(sP1), S0 = lds_addr(sC0), S1 = lds_addr(sC1);

    // Read offsets of the lane: first A / B stage rows and per-slice chunk.
    const int ra = wm * 128 + r, rb = BM + wn * 128 + r;
    const int pa = ra * kSupRowBytes, pb = rb * kSupRowBytes;
    const int x0 = ((0 + hi) ^ (r & 7)) * 16, x1 = ((2 + hi) ^ (r & 7)) * 16;
    const int x2 = ((4 + hi) ^ (r & 7)) * 16, x3 = ((6 + hi) ^ (r & 7)) * 16;

    f32x16_t acc[4][4];
    MxSlice R0, R1;
    uint32_t SC0[8][2], SC1[8][2];

    const int grid = (int)gridDim.x;
    const int nw = (items - (int)blockIdx.x + grid - 1) / grid;
    const int last_it = (int)blockIdx.x + (nw - 1) * grid;
    const bool rot = kStaggerSplit && (blockIdx.x & 1) && nw > 1 && last_it >= sp.Tdp;
    auto item_at = [&](int k) {
        return rot ? (k == 0 ? last_it : (int)blockIdx.x + (k - 1) * grid) : (int)blockIdx.x + k * grid;
    };

    {
        const WorkItem w = work_item(item_at(0), sp, NG);
        const MxSrc q = src_of(w.t);
        L.issue<0, kSupPayLoads, true>(P0, S0, q, w.g0);
        L.issue<0, kSupPayLoads, true>(P1, S1, q, min(w.g0 + 1, w.g1 - 1));
        wait_vmem<kMxLoads>();
        __syncthreads();
    }

    for (int k = 0;; ++k) {
        const int it = item_at(k);
        const WorkItem cur = work_item(it, sp, NG);
        const MxSrc scur = src_of(cur.t);
        const bool has_next = k + 1 < nw;
        const WorkItem nxt = work_item(has_next ? item_at(k + 1) : it, sp, NG);
        const MxSrc snxt = src_of(nxt.t);
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;
        read_mx_slice<0>(R0, sP0, pa, pb, x0);
        read_mx_scales(SC0, sC0, ra, rb, hi);
        // the products are instructions the compiler does not model: keep
        // the accumulator and scale writes above clear of the first ones
        __builtin_amdgcn_sched_barrier(0);
        asm volatile("s_nop 4" ::: "memory");
        __builtin_amdgcn_sched_barrier(0);
        const int gshift = has_next ? nxt.g0 - cur.g1 : -1;
        const int gclamp = has_next ? 0x7FFFFFFF : cur.g1 - 1;

        auto issue_for = [&](auto I0c, auto I1c, auto SCk, uint32_t ldP, uint32_t ldS, int Gt) {
            constexpr int I0v = decltype(I0c)::value, I1v = decltype(I1c)::value;
            constexpr bool SCv = decltype(SCk)::value;
            const bool in_cur = Gt < cur.g1;
            const int Gl = in_cur ? Gt : min(Gt + gshift, gclamp);
            MxSrc q;
            q.off0 = in_cur ? scur.off0 : snxt.off0;
#pragma unroll
            for (int u = 0; u < 4; ++u) q.so[u] = in_cur ? scur.so[u] : snxt.so[u];
            L.issue<I0v, I1v, SCv>(ldP, ldS, q, Gl);
        };

        // One slice: 16 products on the current slice while the next slice
        // (or, at slice 3, after the stage barrier, the next stage's slice 0
        // and scales) is read and, at slice 3, the loads of stage G+2 go out.
        auto slice = [&](auto SLc, int G, const uint8_t* Pc, const uint8_t* Pn, const uint8_t* Sn,
                         uint32_t ldP, uint32_t ldS, MxSlice& Rc, MxSlice& Rn, uint32_t (&SCc)[8][2],
                         uint32_t (&SCn)[8][2]) {
            constexpr int SL = decltype(SLc)::value;
            using Z = std::integral_constant<int, 0>;
            using C8 = std::integral_constant<int, 8>;
            using CP = std::integral_constant<int, kSupPayLoads>;
            using F = std::integral_constant<bool, false>;
            using T = std::integral_constant<bool, true>;
            if (SL == 3) {
                wait_vmem<0>();
                __syncthreads();
                read_mx_slice<0>(Rn, Pn, pa, pb, x0);
                read_mx_scales(SCn, Sn, ra, rb, hi);
                issue_for(Z{}, C8{}, F{}, ldP, ldS, G + 2);
            } else {
                read_mx_slice<SL + 1>(Rn, Pc, pa, pb, SL == 0 ? x1 : (SL == 1 ? x2 : x3));
            }
            mfma_mx16<SL>(acc, Rc, SCc);
            if (SL == 3) {
                issue_for(C8{}, CP{}, T{}, ldP, ldS, G + 2);
                // The products are instructions the compiler does not model:
                // whatever it places after a stage (spills of accumulators,
                // the epilogue) must not read them before the last ones have
                // landed.  The wait overlaps the queued products.
                asm volatile("s_nop 15\n\ts_nop 15\n\ts_nop 15" ::: "memory");
            }
            __builtin_amdgcn_sched_barrier(0);
        };
        using I0 = std::integral_constant<int, 0>;
        using I1 = std::integral_constant<int, 1>;
        using I2 = std::integral_constant<int, 2>;
        using I3 = std::integral_constant<int, 3>;
        // stage scales alternate between SC0 (even stages) and SC1 (odd)
        auto stage = [&](int G, const uint8_t* Pc, const uint8_t* Pn, const uint8_t* Sn, uint32_t ldP,
                         uint32_t ldS, uint32_t (&SCc)[8][2], uint32_t (&SCn)[8][2]) {
            slice(I0{}, G, Pc, Pn, Sn, ldP, ldS, R0, R1, SCc, SCn);
            slice(I1{}, G, Pc, Pn, Sn, ldP, ldS, R1, R0, SCc, SCn);
            slice(I2{}, G, Pc, Pn, Sn, ldP, ldS, R0, R1, SCc, SCn);
            slice(I3{}, G, Pc, Pn, Sn, ldP, ldS, R1, R0, SCc, SCn);
        };
        int G = cur.g0;
        for (; G + 1 < cur.g1; G += 2) {
            stage(G, sP0, sP1, sC1, P0, S0, SC0, SC1);
            stage(G + 1, sP1, sP0, sC0, P1, S1, SC1, SC0);
        }
        if (G < cur.g1) stage(G, sP0, sP1, sC1, P0, S0, SC0, SC1);   // odd stage count (single item)

        // the products above are instructions the compiler does not model:
        // give the last ones time to land before their results are read
        __builtin_amdgcn_sched_barrier(0);
        asm volatile("s_nop 15\n\ts_nop 15\n\ts_nop 15" ::: "memory");
        __builtin_amdgcn_sched_barrier(0);
        store_item<OUT_BF16, VEC>(acc, cur, sp, M, N, tiles_m, tiles_n, wave, lane, a_dec[0] * b_dec[0], C,
                                  sE + wave * kEpiBytes);
        if (!has_next) break;
    }
    wait_vmem<0>();                                  // no load outlives the kernel's LDS
}

// Sum of the partials of the split tiles, in part order, times alpha, into C.
// 64 workgroups per split tile, one per (wave block wv, accumulator (i, j)):
// thread t covers row t/8 of that 32 x 32 block and its 4 columns 4(t%8)..+3,
// so that 8 adjacent threads store 8 adjacent runs of one row.
template <int BMODE, bool OUT_BF16>
__global__ __launch_bounds__(256) void gemm_split_sum_kernel(
    int64_t M, int64_t N, int tiles_m, int tiles_n, SplitPlan sp, const float* __restrict__ a_dec,
    const float* __restrict__ b_dec, void* __restrict__ C, float amul) {
    const int j = blockIdx.x >> 6, wv = (blockIdx.x >> 4) & 3, ij = blockIdx.x & 15;
    int64_t m0, n0;
    tile_origin(sp.Tdp + j, tiles_m, tiles_n, m0, n0);
    const float alpha = (a_dec[0] * b_dec[0]) * amul;
    const int row = threadIdx.x >> 3, c4 = threadIdx.x & 7;     // c4 = 2 g + lane half
    const int lane = row + 32 * (c4 & 1), g = c4 >> 1;
    const float* base = sp.part + (int64_t)j * sp.parts * 65536 + (int64_t)wv * 16384 +
                        ((ij * 4 + g) * 64 + lane) * 4;
    float4 v = *reinterpret_cast<const float4*>(base);
    for (int p = 1; p < sp.parts; ++p) {
        const float4 u = *reinterpret_cast<const float4*>(base + (int64_t)p * 65536);
        v.x += u.x; v.y += u.y; v.z += u.z; v.w += u.w;
    }
    const int64_t m = m0 + (wv >> 1) * 128 + (ij >> 2) * 32 + row;
    const int64_t n = n0 + (wv & 1) * 128 + (ij & 3) * 32 + 4 * c4;
    if (m >= M) return;
    const float r[4] = {alpha * v.x, alpha * v.y, alpha * v.z, alpha * v.w};
    if (OUT_BF16) {
        uint16_t* dst = reinterpret_cast<uint16_t*>(C) + m * N + n;
        if ((N & 3) == 0 && n + 3 < N) {
            *reinterpret_cast<uint2*>(dst) = make_uint2(pack_bf16x2(r[0], r[1]), pack_bf16x2(r[2], r[3]));
        } else {
            for (int q = 0; q < 4; ++q)
                if (n + q < N) dst[q] = (uint16_t)pack_bf16x2(r[q], 0.0f);
        }
    } else {
        float* dst = reinterpret_cast<float*>(C) + m * N + n;
        if ((N & 3) == 0 && n + 3 < N) {
            *reinterpret_cast<float4*>(dst) = make_float4(r[0], r[1], r[2], r[3]);
        } else {
            for (int q = 0; q < 4; ++q)
                if (n + q < N) dst[q] = r[q];
        }
    }
}

hipError_t split_workspace(hipStream_t s, size_t part_floats, float** part) {
    void* p = nullptr;
    const hipError_t e = stream_workspace(kWsSplit, s, part_floats * sizeof(float), &p);
    *part = static_cast<float*>(p);
    return e;
}

// Block-32 scale codes to the block-16 layout the decode kernels read:
// out[r][j] = in[r / rrep][j / 2] (rrep 2 for 32 x 32 tile scales, whose
// tile rows cover two 16-row tile rows).
__global__ __launch_bounds__(256) void expand_scales_kernel(const uint8_t* __restrict__ in, int64_t cols_in,
                                                            int rrep, uint8_t* __restrict__ out,
                                                            int64_t rows_out, int64_t cols_out) {
    const int64_t n = rows_out * cols_out;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
        const int64_t r = i / cols_out, j = i - r * cols_out;
        out[i] = in[(r / rrep) * cols_in + j / 2];
    }
}

hipError_t expand_scales(const uint8_t* in, int64_t cols_in, int rrep, uint8_t* out, int64_t rows_out,
                         int64_t cols_out, hipStream_t s) {
    const int64_t n = rows_out * cols_out;
    if (n <= 0) return hipSuccess;
    const int64_t blocks = min((n + 255) / 256, (int64_t)4096);
    hipLaunchKernelGGL(expand_scales_kernel, dim3((unsigned)blocks), dim3(256), 0, s, in, cols_in, rrep, out,
                       rows_out, cols_out);
    return hipGetLastError();
}

constexpr int kSplitRemDiv = 2;

// Whether the whole-tile epilogue may store vector runs: N a multiple of the
// run (8 bf16 or 4 fp32 columns), and for bf16 every row offset of the padded
// tile grid below 2^31 bytes, since that path drops rows past M by their
// offset alone (lane base + uniform row offset, no row compare).
template <bool OUT_BF16>
bool vector_epilogue(int64_t N, int tiles_m) {
    if (OUT_BF16) return N % 8 == 0 && (int64_t)tiles_m * BM * N * 2 < ((int64_t)1 << 31);
    return N % 4 == 0;
}

template <int BMODE, bool OUT_BF16>
hipError_t launch_reg(int64_t M, int64_t N, int64_t K, const uint8_t* a, const uint8_t* as,
                      const float* ad, const uint8_t* b, const uint8_t* bs, const float* bd,
                      void* c, float amul, hipStream_t s, const FixedScratch* fx) {
    const int tiles_m = (int)((M + BM - 1) / BM);
    const int tiles_n = (int)((N + BN - 1) / BN);
    const int T = tiles_m * tiles_n;
    const int NG = (int)(K / (kSupK * BK));
    int dev = 0, cus = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    // One workgroup per CU at a time (LDS-bound).  Split only a partial last
    // wave of tiles that leaves at least 1 - 1/kSplitRemDiv of the CUs idle;
    // parts cover whole stage pairs when the stage count is even.
    const bool even = NG % 2 == 0;
    SplitPlan sp{T, 1, nullptr};
    const int rem = cus > 0 ? T % cus : 0;
    if (T > cus && rem > 0 && rem <= cus / kSplitRemDiv) {
        const int parts = min(cus / rem, even ? NG / 2 : NG);
        if (parts > 1) {
            sp.Tdp = T - rem;
            sp.parts = parts;
            const size_t need = (size_t)rem * parts * 65536;
            if (fx != nullptr) {
                // caller-supplied buffer: the same plan, or a refusal
                if (need > fx->floats) return hipErrorOutOfMemory;
                sp.part = fx->part;
            } else {
                e = split_workspace(s, need, &sp.part);
                if (e != hipSuccess) return e;
            }
        }
    }
    const int items = sp.Tdp + (T - sp.Tdp) * sp.parts;
    // persistent (one workgroup per CU walking the items) when every item has
    // an even stage count, else one item per workgroup
    const int grid = (even && cus > 0) ? min(items, cus) : items;
    if (vector_epilogue<OUT_BF16>(N, tiles_m))
        hipLaunchKernelGGL((gemm_fp4_reg_kernel<BMODE, OUT_BF16, true>), dim3((unsigned)grid), dim3(kGemmThreads),
                           0, s, (int)M, (int)N, (int)K, tiles_m, tiles_n, items, sp, a, as, ad, b, bs, bd, c, amul);
    else
        hipLaunchKernelGGL((gemm_fp4_reg_kernel<BMODE, OUT_BF16, false>), dim3((unsigned)grid), dim3(kGemmThreads),
                           0, s, (int)M, (int)N, (int)K, tiles_m, tiles_n, items, sp, a, as, ad, b, bs, bd, c, amul);
    if ((e = hipGetLastError()) != hipSuccess || sp.parts == 1) return e;
    hipLaunchKernelGGL((gemm_split_sum_kernel<BMODE, OUT_BF16>), dim3((unsigned)(64 * (T - sp.Tdp))), dim3(256),
                       0, s, M, N, tiles_m, tiles_n, sp, ad, bd, c, amul);
    return hipGetLastError();
}

template <bool OUT_BF16>
hipError_t launch_mx(int64_t M, int64_t N, int64_t K, const uint8_t* a, const uint8_t* as,
                     const float* ad, const uint8_t* b, const uint8_t* bs, const float* bd,
                     void* c, hipStream_t s) {
    const int tiles_m = (int)((M + BM - 1) / BM);
    const int tiles_n = (int)((N + BN - 1) / BN);
    const int T = tiles_m * tiles_n;
    const int NG = (int)(K / (kSupK * BK));
    int dev = 0, cus = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    const bool even = NG % 2 == 0;
    SplitPlan sp{T, 1, nullptr};
    const int rem = cus > 0 ? T % cus : 0;
    if (T > cus && rem > 0 && rem <= cus / kSplitRemDiv) {
        const int parts = min(cus / rem, even ? NG / 2 : NG);
        if (parts > 1) {
            sp.Tdp = T - rem;
            sp.parts = parts;
            e = split_workspace(s, (size_t)rem * parts * 65536, &sp.part);
            if (e != hipSuccess) return e;
        }
    }
    const int items = sp.Tdp + (T - sp.Tdp) * sp.parts;
    const int grid = (even && cus > 0) ? min(items, cus) : items;
    if (vector_epilogue<OUT_BF16>(N, tiles_m))
        hipLaunchKernelGGL((gemm_mx_kernel<OUT_BF16, true>), dim3((unsigned)grid), dim3(kGemmThreads), 0, s, (int)M,
                           (int)N, (int)K, tiles_m, tiles_n, items, sp, a, as, ad, b, bs, bd, c);
    else
        hipLaunchKernelGGL((gemm_mx_kernel<OUT_BF16, false>), dim3((unsigned)grid), dim3(kGemmThreads), 0, s,
                           (int)M, (int)N, (int)K, tiles_m, tiles_n, items, sp, a, as, ad, b, bs, bd, c);
    if ((e = hipGetLastError()) != hipSuccess || sp.parts == 1) return e;
    hipLaunchKernelGGL((gemm_split_sum_kernel<(int)BScale::Row, OUT_BF16>), dim3((unsigned)(64 * (T - sp.Tdp))),
                       dim3(256), 0, s, M, N, tiles_m, tiles_n, sp, ad, bd, c, 1.0f);
    return hipGetLastError();
}

template <int BMODE, bool OUT_BF16, bool FULLK>
hipError_t launch_one(int64_t M, int64_t N, int64_t K, const uint8_t* a, const uint8_t* as,
                      const float* ad, const uint8_t* b, const uint8_t* bs, const float* bd,
                      void* c, float amul, hipStream_t s) {
    // the dynamic LDS attribute, set once per device (setting it twice, when
    // two threads race here, is harmless)
    static std::atomic<uint64_t> attr_set{0};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    const uint64_t bit = (uint64_t)1 << (dev & 63);
    if ((attr_set.load(std::memory_order_acquire) & bit) == 0) {
        e = hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_fp4_kernel<BMODE, OUT_BF16, FULLK>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, kSmemBytes);
        if (e != hipSuccess) return e;
        attr_set.fetch_or(bit, std::memory_order_release);
    }
    const int tiles_m = (int)((M + BM - 1) / BM);
    const int tiles_n = (int)((N + BN - 1) / BN);
    hipLaunchKernelGGL((gemm_fp4_kernel<BMODE, OUT_BF16, FULLK>),
                       dim3((unsigned)(tiles_m * tiles_n)), dim3(kGemmThreads), kSmemBytes, s, M,
                       N, K, tiles_m, tiles_n, a, as, ad, b, bs, bd, c, amul);
    return hipGetLastError();
}

template <int BMODE>
hipError_t launch_mode(int64_t M, int64_t N, int64_t K, const uint8_t* a, const uint8_t* as,
                       const float* ad, const uint8_t* b, const uint8_t* bs, const float* bd,
                       void* c, bool c_bf16, float amul, hipStream_t s, const FixedScratch* fx) {
    // the register-decode kernel addresses operands and C with 32-bit offsets
    const int64_t kLim = (int64_t)1 << 31;
    if (K % (4 * BK) == 0 && K > 0 && M * (K / 2) < kLim && N * (K / 2) < kLim && M * N * 4 < kLim)
        return c_bf16 ? launch_reg<BMODE, true>(M, N, K, a, as, ad, b, bs, bd, c, amul, s, fx)
                      : launch_reg<BMODE, false>(M, N, K, a, as, ad, b, bs, bd, c, amul, s, fx);
    if (K % BK == 0 && K > 0)
        return c_bf16 ? launch_dma<BMODE, true>(M, N, K, a, as, ad, b, bs, bd, c, amul, s)
                      : launch_dma<BMODE, false>(M, N, K, a, as, ad, b, bs, bd, c, amul, s);
    return c_bf16 ? launch_one<BMODE, true, false>(M, N, K, a, as, ad, b, bs, bd, c, amul, s)
                  : launch_one<BMODE, false, false>(M, N, K, a, as, ad, b, bs, bd, c, amul, s);
}

}  // namespace

hipError_t launch_gemm(BScale bmode, float amul, int64_t M, int64_t N, int64_t K, const uint8_t* a,
                       const uint8_t* a_scales, const float* a_dec, const uint8_t* b,
                       const uint8_t* b_scales, const float* b_dec, void* c, bool c_bf16,
                       hipStream_t s, const FixedScratch* fx) {
    if (M == 0 || N == 0) return hipSuccess;
    switch (bmode) {
        case BScale::Row:
            return launch_mode<(int)BScale::Row>(M, N, K, a, a_scales, a_dec, b, b_scales, b_dec, c, c_bf16, amul, s,
                                                 fx);
        case BScale::Tile:
            return launch_mode<(int)BScale::Tile>(M, N, K, a, a_scales, a_dec, b, b_scales, b_dec, c, c_bf16, amul,
                                                  s, fx);
        case BScale::TileDgrad:
            return launch_mode<(int)BScale::TileDgrad>(M, N, K, a, a_scales, a_dec, b, b_scales, b_dec, c, c_bf16,
                                                       amul, s, fx);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_gemm_b32(BScale bmode, float amul, bool pm, float grid_d, int64_t M, int64_t N, int64_t K,
                           const uint8_t* a, const uint8_t* a_scales, const float* a_dec, const uint8_t* b,
                           const uint8_t* b_scales, const float* b_dec, void* c, bool c_bf16, hipStream_t s) {
    const uint8_t* as16 = a_scales;
    const uint8_t* bs16 = b_scales;
    if (M > 0 && N > 0 && K > 0) {
        const bool tiled = bmode != BScale::Row;
        const int64_t kb16 = K / 16, kb32 = K / 32;
        const int64_t brows16 = tiled ? N / 16 : N;
        const size_t abytes = (size_t)((M * kb16 + 255) / 256 * 256);
        const size_t bbytes = (size_t)(brows16 * kb16);
        void* ws = nullptr;
        hipError_t e = stream_workspace(kWsScales, s, abytes + bbytes, &ws);
        if (e != hipSuccess) return e;
        uint8_t* wa = static_cast<uint8_t*>(ws);
        uint8_t* wb = wa + abytes;
        if ((e = expand_scales(a_scales, kb32, 1, wa, M, kb16, s)) != hipSuccess) return e;
        if ((e = expand_scales(b_scales, kb32, tiled ? 2 : 1, wb, brows16, kb16, s)) != hipSuccess) return e;
        as16 = wa;
        bs16 = wb;
    }
    return pm ? launch_gemm_pm(bmode, amul, grid_d, M, N, K, a, as16, a_dec, b, bs16, b_dec, c, c_bf16, s)
              : launch_gemm(bmode, amul, M, N, K, a, as16, a_dec, b, bs16, b_dec, c, c_bf16, s);
}

hipError_t launch_gemm_mx(int64_t M, int64_t N, int64_t K, const uint8_t* a, const uint8_t* a_scales,
                          const float* a_dec, const uint8_t* b, const uint8_t* b_scales,
                          const float* b_dec, void* c, bool c_bf16, hipStream_t s) {
    if (M == 0 || N == 0) return hipSuccess;
    return c_bf16 ? launch_mx<true>(M, N, K, a, a_scales, a_dec, b, b_scales, b_dec, c, s)
                  : launch_mx<false>(M, N, K, a, a_scales, a_dec, b, b_scales, b_dec, c, s);
}

}  // namespace ue5m3
