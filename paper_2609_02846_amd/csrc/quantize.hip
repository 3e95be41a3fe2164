// Block quantizers of the UE5M3 FP4 recipe (paper eq:microscaling,
// eq:scale-target, eq:sr, Table 5).
//
// Per block B of 16 elements (or a 16x16 tile), in binary32 with one
// round-to-nearest-even per operation and no fused operations:
//   a = max |x_B|   (exact integer max on bf16 bits)
//   code = UE5M3(a * S), zero code -> code of 1.0 (zero-scale rule)
//   r = G / UE5M3value(code)
//   nibble_i = E2M1_RN(x_i * r)  or  E2M1_SR(x_i * r, philox word of element i)
// with S = T/g, G = 6T/g computed in every workgroup prologue from the held
// amax g in device memory.
//
// All three kernels are HBM-bound streaming passes: 2 bytes of bf16 read and
// 0.5 + 1/16 (1D) or 0.5 + 1/256 (2D) bytes written per element, plus 0.5
// bytes for the optional transposed weight payload.  HBM is written in
// 64-byte units, so every output is written in runs of at least 64
// contiguous bytes from one store instruction: outputs whose natural
// per-lane piece is smaller (the transposed payloads and scales) are
// assembled in LDS first.
#include <atomic>
#include <type_traits>

#include "codec.hpp"
#include "launch.hpp"
#include "rht.hpp"

namespace ue5m3 {
namespace {

constexpr int kThreads = 256;

struct BlockScale {
    uint32_t code;
    float r;
};

// SR values in the scaled form (S23): the SR conversion divides its input
// by its power-of-two scale operand exactly (checked on gfx950 against the
// unscaled form over every binade of binary32 from 2^-126 up, and for +-inf
// and values whose scaled form overflows: the same nibbles), so an element
// can enter as y 2^23 = x (r 2^23) with scale 2^23.  The bucket check then
// converts |y 2^23| to an integer directly, one multiply fewer per element.
// x (r 2^23) equals (x r) 2^23 exactly while x r is a normal binary32 value
// and r 2^23 is finite; a launch takes the scaled form only when
// G <= 2^80, so that r <= G 2^17 keeps r 2^23 finite.  Below 2^-126 (where
// x r has fewer bits) the unscaled threshold is 1 or 0, the element's
// bucket value is then ~w and it is flagged for every w < 1024, which
// includes the one word (w = 0) that could round it up: the software
// rounding redoes it from the exact x r.
constexpr float kS23 = 0x1p23f;
constexpr float kS23MaxG = 0x1p80f;

// Reciprocals G / value(c) of the 256 scale codes in LDS, one per thread of
// the workgroup (kThreads == 256): a block's reciprocal is then one LDS read
// instead of a decode and a division per block.  The table entry is the same
// binary32 division, so the same value.  E8M0 needs no table (r = 2^-E is
// formed exactly from the code).  Ends with a barrier: call it where every
// thread of the workgroup arrives.
template <int FMT>
__device__ __forceinline__ void fill_recip(float* rtab, const Multipliers& m) {
    if (FMT == (int)ScaleKind::E8M0) return;
    const uint32_t c = threadIdx.x;
    rtab[c] = m.G / (FMT == (int)ScaleKind::E4M3 ? e4m3_decode(c) : ue5m3_decode(c));
    __syncthreads();
}

// UE5M3 / E4M3 block scale of a block whose largest magnitude is a (any
// binary32 value, e.g. of a transformed block): code = nearest code of
// a * S (zero code -> code of 1.0), r = G / value(code) from the table.
template <int FMT>
__device__ __forceinline__ BlockScale block_scale_value(float a, const Multipliers& m, const float* rtab) {
    BlockScale bs;
    const bool e4 = FMT == (int)ScaleKind::E4M3;
    uint32_t code = e4 ? e4m3_encode(a * m.S) : ue5m3_encode(a * m.S);
    code = code ? code : (e4 ? kE4M3CodeOne : kCodeOne);
    bs.code = code;
    bs.r = rtab[code];
    return bs;
}

// Block scale and reciprocal of a block from the bf16 bits of its largest
// magnitude.  E8M0: the power-of-two exponent of the OCP microscaling rule
// and r = 2^-E (no tensor scale).
template <int FMT>
__device__ __forceinline__ BlockScale block_scale(uint32_t amax_bits15, const Multipliers& m,
                                                  const float* rtab) {
    if (FMT == (int)ScaleKind::E8M0) {
        BlockScale bs;
        bs.code = e8m0_code_of_amax(amax_bits15);
        bs.r = e8m0_reciprocal(bs.code);
        return bs;
    }
    return block_scale_value<FMT>(__uint_as_float(amax_bits15 << 16), m, rtab);
}

// Packed 16-bit unsigned maximum (per half).
__device__ __forceinline__ uint32_t pk_max_u16(uint32_t a, uint32_t b) {
    uint32_t r;
    asm("v_pk_max_u16 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
    return r;
}

// Tensor multipliers of a quantizer launch (E8M0 has no tensor scale: the
// held amax is not read and the decode multiplier is 1).
template <int FMT>
__device__ __forceinline__ Multipliers kernel_multipliers(const float* amax_dev, float T) {
    if (FMT == (int)ScaleKind::E8M0) {
        Multipliers m;
        m.S = 1.0f;
        m.G = 1.0f;
        m.dec = 1.0f;
        return m;
    }
    return tensor_multipliers(*amax_dev, T);
}

// E2M1 round-to-nearest-even of y0, y1 into byte SEL of p (y0 in the low
// nibble).  The gfx950 conversion with scale 1.0 is exactly the E2M1 RNE of
// the binary32 input with saturation to code 7 at |y| >= 6 and the sign in
// bit 3 (including -0), identical to the E2M1 RNE definition for all 2^32
// inputs.
template <int SEL>
__device__ __forceinline__ uint32_t rn_pair(uint32_t p, float y0, float y1) {
    return __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(p, y0, y1, 1.0f, SEL);
}

// E2M1 stochastic rounding on the gfx950 SR pair conversion.  For a pair
// (y0, y1) and random operand R the instruction rounds y0 with bits 31..10
// of R and y1 with bits 30..9; with R = ~w (y0) it rounds up iff
// (w >> 10) < floor(frac * 2^22), while the rule here (w < ceil(frac * 2^32))
// uses all 32 bits.  The two agree except when |y| < 1 and w >> 10 equals
// floor(frac * 2^22) -- the 1024 words around the threshold -- which the
// bucket check below flags.
// (For |y| >= 1, frac * 2^32 is a multiple of 1024 and the rules coincide.)
// Each pair is converted twice, once with each element's own word placed
// where that element reads it, and the two valid nibbles are merged.  The
// words arrive complemented (nw = ~w, sr_nwords4).  A group with a flagged
// element has all its nibbles redone by the software rounding.
typedef float v2f_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

// Written as an instruction with p as a read-write operand: the compiler's
// builtin for this conversion does not keep the destination's other bytes.
// S23: the pair arrives scaled by 2^23 and the conversion divides it back.
template <int SEL, bool S23 = false>
__device__ __forceinline__ uint32_t sr_pair(uint32_t p, v2f_t v, uint32_t r) {
    if (S23) {
        const float sc = kS23;
        if (SEL == 0) asm("v_cvt_scalef32_sr_pk_fp4_f32 %0, %1, %2, %3" : "+v"(p) : "v"(v), "v"(r), "s"(sc));
        if (SEL == 1) asm("v_cvt_scalef32_sr_pk_fp4_f32 %0, %1, %2, %3 op_sel:[0,0,1,0]" : "+v"(p) : "v"(v), "v"(r), "s"(sc));
        if (SEL == 2) asm("v_cvt_scalef32_sr_pk_fp4_f32 %0, %1, %2, %3 op_sel:[0,0,0,1]" : "+v"(p) : "v"(v), "v"(r), "s"(sc));
        if (SEL == 3) asm("v_cvt_scalef32_sr_pk_fp4_f32 %0, %1, %2, %3 op_sel:[0,0,1,1]" : "+v"(p) : "v"(v), "v"(r), "s"(sc));
        return p;
    }
    if (SEL == 0) asm("v_cvt_scalef32_sr_pk_fp4_f32 %0, %1, %2, 1.0" : "+v"(p) : "v"(v), "v"(r));
    if (SEL == 1) asm("v_cvt_scalef32_sr_pk_fp4_f32 %0, %1, %2, 1.0 op_sel:[0,0,1,0]" : "+v"(p) : "v"(v), "v"(r));
    if (SEL == 2) asm("v_cvt_scalef32_sr_pk_fp4_f32 %0, %1, %2, 1.0 op_sel:[0,0,0,1]" : "+v"(p) : "v"(v), "v"(r));
    if (SEL == 3) asm("v_cvt_scalef32_sr_pk_fp4_f32 %0, %1, %2, 1.0 op_sel:[0,0,1,1]" : "+v"(p) : "v"(v), "v"(r));
    return p;
}

// Bucket value of y and its complemented word nw: with q = floor(|y| 2^23)
// (the conversion to integer saturates: |y| 2^23 may exceed 2^32) and
// A = (q mod 2^22) * 1024 = q << 10 (mod 2^32), w >> 10 equals q mod 2^22
// exactly when w lies in [A, A + 1023], i.e. when A + nw = A - w - 1
// (mod 2^32) is one of the top 1024 values.  An element is flagged when its
// bucket value exceeds kBucketTop: the 1024 words around y's threshold for
// |y| < 1, or spuriously with probability 2^-22 (|y| >= 1), which only
// costs a redo.  A group tests the maximum of its bucket values once.
constexpr uint32_t kBucketTop = 0xFFFFFBFFu;
// S23: y arrives as y 2^23 (the product the conversion takes).
template <bool S23 = false>
__device__ __forceinline__ uint32_t sr_bucket(float y, uint32_t nw) {
    uint32_t q;
    if (S23)
        asm("v_cvt_u32_f32_e64 %0, |%1|" : "=v"(q) : "v"(y));
    else
        asm("v_cvt_u32_f32 %0, %1" : "=v"(q) : "v"(fabsf(y) * 0x1p23f));
    uint32_t t;
    asm("v_lshl_add_u32 %0, %1, 10, %2" : "=v"(t) : "v"(q), "v"(nw));
    return t;
}

// 8 values y (element e -> nibble e) by SR with complemented words nw.
// S23: y holds the scaled values and exact(e) gives element e's unscaled
// binary32 value for the software rounding.
template <bool S23, typename Exact>
__device__ __forceinline__ uint32_t sr8(const float (&y)[8], const uint32_t* nw, Exact exact) {
    uint32_t lo = 0u, hi = 0u;                 // valid low / high nibbles
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const v2f_t v = {y[2 * k], y[2 * k + 1]};
        const uint32_t r0 = nw[2 * k];
        const uint32_t r1 = __builtin_amdgcn_alignbit(nw[2 * k + 1], nw[2 * k + 1], 1);
        if (k == 0) { lo = sr_pair<0, S23>(lo, v, r0); hi = sr_pair<0, S23>(hi, v, r1); }
        if (k == 1) { lo = sr_pair<1, S23>(lo, v, r0); hi = sr_pair<1, S23>(hi, v, r1); }
        if (k == 2) { lo = sr_pair<2, S23>(lo, v, r0); hi = sr_pair<2, S23>(hi, v, r1); }
        if (k == 3) { lo = sr_pair<3, S23>(lo, v, r0); hi = sr_pair<3, S23>(hi, v, r1); }
    }
    uint32_t p = (lo & 0x0F0F0F0Fu) | (hi & 0xF0F0F0F0u);
    uint32_t tb = 0u;
#pragma unroll
    for (int e = 0; e < 8; ++e) tb = max(tb, sr_bucket<S23>(y[e], nw[e]));
    if (tb > kBucketTop) {
        p = 0u;
#pragma unroll
        for (int e = 0; e < 8; ++e) p |= e2m1_sr(S23 ? exact(e) : y[e], ~nw[e]) << (4 * e);
    }
    return p;
}

template <bool S23 = false>
__device__ __forceinline__ uint32_t sr8(const float (&y)[8], const uint32_t* nw) {
    static_assert(!S23, "the scaled form needs the exact values");
    return sr8<false>(y, nw, [&](int e) { return y[e]; });
}

// 4 values y (element e -> nibble e of the low 16 bits) by SR with
// complemented words nw.
__device__ __forceinline__ uint32_t sr4(const float (&y)[4], const uint32_t* nw) {
    uint32_t lo = 0u, hi = 0u;
    const v2f_t v0 = {y[0], y[1]}, v1 = {y[2], y[3]};
    lo = sr_pair<0>(lo, v0, nw[0]);
    hi = sr_pair<0>(hi, v0, __builtin_amdgcn_alignbit(nw[1], nw[1], 1));
    lo = sr_pair<1>(lo, v1, nw[2]);
    hi = sr_pair<1>(hi, v1, __builtin_amdgcn_alignbit(nw[3], nw[3], 1));
    uint32_t p = (lo & 0x0F0Fu) | (hi & 0xF0F0u);
    const uint32_t tb = max(max(sr_bucket(y[0], nw[0]), sr_bucket(y[1], nw[1])),
                            max(sr_bucket(y[2], nw[2]), sr_bucket(y[3], nw[3])));
    if (tb > kBucketTop) {
        p = 0u;
#pragma unroll
        for (int e = 0; e < 4; ++e) p |= e2m1_sr(y[e], ~nw[e]) << (4 * e);
    }
    return p;
}

// Quantize the 8 bf16 values held in v (element e in half e&1 of word e>>1)
// with reciprocal r; returns 8 nibbles packed little-endian.  For SR, w holds
// the 8 complemented Philox words of the elements; S23: the SR values are
// formed scaled, as x (r 2^23).
template <bool SR, bool S23 = false>
__device__ __forceinline__ uint32_t quant8(const uint4& v, float r, const uint32_t* w) {
    const uint32_t vv[4] = {v.x, v.y, v.z, v.w};
    if (!SR) {
        uint32_t p = 0;
        p = rn_pair<0>(p, bf16_lo(vv[0]) * r, bf16_hi(vv[0]) * r);
        p = rn_pair<1>(p, bf16_lo(vv[1]) * r, bf16_hi(vv[1]) * r);
        p = rn_pair<2>(p, bf16_lo(vv[2]) * r, bf16_hi(vv[2]) * r);
        p = rn_pair<3>(p, bf16_lo(vv[3]) * r, bf16_hi(vv[3]) * r);
        return p;
    }
    auto xe = [&](int e) { return (e & 1) ? bf16_hi(vv[e >> 1]) : bf16_lo(vv[e >> 1]); };
    const float ry = S23 ? r * kS23 : r;
    float y[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) y[e] = xe(e) * ry;
    return sr8<S23>(y, w, [&](int e) { return xe(e) * r; });
}

// Column-wise nibbles of 16 rows of one column (values v[r] * r_, rows in
// order) into two words, RN or SR (w: complemented Philox words).
template <bool SR>
__device__ __forceinline__ void quant_col16(const float (&xv)[16], float r_, const uint32_t (&w)[16],
                                            uint32_t& p0, uint32_t& p1) {
    if (!SR) {
        p0 = 0u;
        p1 = 0u;
        p0 = rn_pair<0>(p0, xv[0] * r_, xv[1] * r_);
        p0 = rn_pair<1>(p0, xv[2] * r_, xv[3] * r_);
        p0 = rn_pair<2>(p0, xv[4] * r_, xv[5] * r_);
        p0 = rn_pair<3>(p0, xv[6] * r_, xv[7] * r_);
        p1 = rn_pair<0>(p1, xv[8] * r_, xv[9] * r_);
        p1 = rn_pair<1>(p1, xv[10] * r_, xv[11] * r_);
        p1 = rn_pair<2>(p1, xv[12] * r_, xv[13] * r_);
        p1 = rn_pair<3>(p1, xv[14] * r_, xv[15] * r_);
        return;
    }
    float y0[8], y1[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        y0[k] = xv[k] * r_;
        y1[k] = xv[8 + k] * r_;
    }
    p0 = sr8(y0, w);
    p1 = sr8(y1, w + 8);
}

// Packed 16-bit maxima of |x| over the 8 bf16 values of v, into acc.
__device__ __forceinline__ uint32_t amax8_pk(const uint4& v, uint32_t acc) {
    acc = pk_max_u16(acc, v.x & 0x7FFF7FFFu);
    acc = pk_max_u16(acc, v.y & 0x7FFF7FFFu);
    acc = pk_max_u16(acc, v.z & 0x7FFF7FFFu);
    return pk_max_u16(acc, v.w & 0x7FFF7FFFu);
}

// Philox words of elements 4j .. 4j+3 for the 4 columns c..c+3 of one row,
// element index e0 = row * cols + c (even).  When e0 % 4 == 0 one Philox
// block holds them; otherwise (cols % 4 == 2) they straddle two blocks.
template <bool ALIGNED = false>
__device__ __forceinline__ void words4(uint64_t e0, uint32_t tid, uint32_t k0, uint32_t k1,
                                       uint32_t* w) {
    const uint4 a = sr_words4(e0 >> 2, tid, k0, k1);
    if (ALIGNED || (e0 & 3) == 0) {
        w[0] = a.x; w[1] = a.y; w[2] = a.z; w[3] = a.w;
    } else {
        const uint4 b = sr_words4((e0 >> 2) + 1, tid, k0, k1);
        w[0] = a.z; w[1] = a.w; w[2] = b.x; w[3] = b.y;
    }
}

// The same four words complemented (~w, the SR operand form).
template <bool ALIGNED = false>
__device__ __forceinline__ void nwords4(uint64_t e0, uint32_t tid, uint32_t k0, uint32_t k1,
                                        uint32_t* nw) {
    const uint4 a = sr_nwords4(e0 >> 2, tid, k0, k1);
    if (ALIGNED || (e0 & 3) == 0) {
        nw[0] = a.x; nw[1] = a.y; nw[2] = a.z; nw[3] = a.w;
    } else {
        const uint4 b = sr_nwords4((e0 >> 2) + 1, tid, k0, k1);
        nw[0] = a.z; nw[1] = a.w; nw[2] = b.x; nw[3] = b.y;
    }
}

// ------------------------------------------------------------ rows (1D) --
// The flat tensor is a sequence of blocks of 16 (32: E8M0, block-size-32
// control) elements.  One
// lane per block: two (four) 16-byte loads, 8 (16) bytes of payload and 1
// byte of scale, so one wave instruction stores 512 (1024) contiguous payload
// bytes and 64 scale bytes.  Persistent grid: a lane walks blocks b,
// b + stride, ..., loading the next block before quantizing the current one.
// H: 16-element halves per block (2 for E8M0 and for the block-size-32
// control of UE5M3 / E4M3).
template <bool SR, int FMT, int H>
__global__ __launch_bounds__(kThreads) void quant_rows_kernel(
    const uint4* __restrict__ x, int64_t nblocks, const float* __restrict__ amax_dev, float T,
    uint32_t key0, uint32_t key1, uint32_t tid, uint2* __restrict__ payload,
    uint8_t* __restrict__ scales, float* __restrict__ dec_out) {
    static_assert(FMT != (int)ScaleKind::E8M0 || H == 2, "E8M0 blocks are 32");
    __shared__ float rtab[256];
    const Multipliers m = kernel_multipliers<FMT>(amax_dev, T);
    if (dec_out != nullptr && blockIdx.x == 0 && threadIdx.x == 0) *dec_out = m.dec;
    fill_recip<FMT>(rtab, m);
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    // S23: the scaled SR form (a uniform choice per launch, see kS23MaxG)
    auto run = [&](auto S23c) {
        constexpr bool S23 = decltype(S23c)::value;
        int64_t b = (int64_t)blockIdx.x * kThreads + threadIdx.x;
        uint4 c[2 * H];
        if (b < nblocks) {
#pragma unroll
            for (int i = 0; i < 2 * H; ++i) c[i] = x[2 * H * b + i];
        }
        for (; b < nblocks; b += stride) {
            const int64_t bn = b + stride;
            uint4 n[2 * H];
#pragma unroll
            for (int i = 0; i < 2 * H; ++i) n[i] = make_uint4(0u, 0u, 0u, 0u);
            if (bn < nblocks) {
#pragma unroll
                for (int i = 0; i < 2 * H; ++i) n[i] = x[2 * H * bn + i];
            }
            uint32_t mp = 0u;
#pragma unroll
            for (int i = 0; i < 2 * H; ++i) mp = amax8_pk(c[i], mp);
            const BlockScale bs = block_scale<FMT>(max(mp & 0xFFFFu, mp >> 16), m, rtab);
#pragma unroll
            for (int h = 0; h < H; ++h) {
                // elements 16(Hb + h) .. +15: Philox blocks 4(Hb + h) .. +3,
                // made per half of 8 so that only 8 words are live at a time
                uint32_t out[2];
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    uint32_t nw[8];
                    if (SR) {
#pragma unroll
                        for (int i = 0; i < 2; ++i) {
                            const uint4 q = sr_nwords4((uint64_t)(H * b + h) * 4 + 2 * u + i, tid, key0, key1);
                            nw[4 * i] = q.x; nw[4 * i + 1] = q.y; nw[4 * i + 2] = q.z; nw[4 * i + 3] = q.w;
                        }
                    }
                    out[u] = quant8<SR, S23>(c[2 * h + u], bs.r, nw);
                    if (SR) __builtin_amdgcn_sched_barrier(0);
                }
                payload[H * b + h] = make_uint2(out[0], out[1]);
            }
            scales[b] = (uint8_t)bs.code;
#pragma unroll
            for (int i = 0; i < 2 * H; ++i) c[i] = n[i];
        }
    };
    if (SR && FMT != (int)ScaleKind::E8M0 && m.G <= kS23MaxG)
        run(std::integral_constant<bool, SR && FMT != (int)ScaleKind::E8M0>{});
    else
        run(std::false_type{});
}

// Tiles of the 2D and dual-axis quantizers: 128 columns x 8 tile rows of 16.
constexpr int kTileCols = 128;
constexpr int kTileRowTiles = 8;

// The 64-byte runs of a transposed payload assembled in LDS, laid out
// [tile row][column] (st[k][8 c .. 8 c + 7]: the 8 bytes of 16-row tile row
// k of column cw + c, so that each lane writes its 4 columns of one tile row
// as one contiguous 32-byte piece, free of bank conflicts), written to
// dst[(cw + c) * ld + off ...]: four adjacent lanes write one column's run as
// 16-byte pieces, so one store instruction writes 16 whole 64-byte runs.
// nvalid: tile rows inside the tensor; a run that is not whole, or a row
// stride that is not a multiple of 16, goes out as 8-byte pieces.
__device__ __forceinline__ void store_cols64(const uint8_t (*st)[kTileCols * 8], uint8_t* __restrict__ dst,
                                             int64_t cw, int64_t cols, int64_t ld, int64_t off, int nvalid,
                                             int t) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const int chunk = t + kThreads * u;
        const int col = chunk >> 2, part = chunk & 3;
        const int64_t gc = cw + col;
        if (col >= kTileCols || gc >= cols) continue;
        uint8_t* d = dst + gc * ld + off + part * 16;
        const uint2 a = *reinterpret_cast<const uint2*>(&st[2 * part][col * 8]);
        const uint2 b = *reinterpret_cast<const uint2*>(&st[2 * part + 1][col * 8]);
        if (nvalid == kTileRowTiles && (ld & 15) == 0) {
            *reinterpret_cast<uint4*>(d) = make_uint4(a.x, a.y, b.x, b.y);
        } else {
            if (2 * part < nvalid) *reinterpret_cast<uint2*>(d) = a;
            if (2 * part + 1 < nvalid) *reinterpret_cast<uint2*>(d + 8) = b;
        }
    }
}

// A lane's 4 adjacent columns c = 4q .. 4q+3 of one tile row (pk[j][0..1]:
// 8 payload bytes of column 4q + j) into the staging row st (see
// store_cols64): one contiguous 32-byte piece.
__device__ __forceinline__ void stage_cols4(uint8_t* st, int q, const uint32_t (&pk)[4][2]) {
    uint4* d = reinterpret_cast<uint4*>(st + 32 * q);
    d[0] = make_uint4(pk[0][0], pk[0][1], pk[1][0], pk[1][1]);
    d[1] = make_uint4(pk[2][0], pk[2][1], pk[3][0], pk[3][1]);
}

// ------------------------------------------------ columns (1D, transposed) --
// Blocks are 16 consecutive rows of one column; output is the row blocking
// of x^T: payload_t [cols, rows/2], scales_t [cols, rows/16].
// Work item = 128 columns x a chunk of up to 64 row blocks.  A workgroup
// walks its items (item, item + grid, ...) group by group, a group being 8
// row blocks (thread t handles row block t / 32 of the group; lane
// q = t % 32 holds the 4 adjacent columns 4q .. 4q+3), loading the next group
// -- possibly of its next item -- while it quantizes the current one.  Per
// group each column gains 8 x 8 = 64 payload bytes, assembled in LDS and
// written as whole 64-byte runs (store_cols64); scale bytes collect in LDS over the item
// (up to 64 bytes per column) before they are written.
constexpr int kColCols = 128;
constexpr int kColGroupRB = 8;
static_assert(kColCols == kTileCols && kColGroupRB == kTileRowTiles,
              "the column quantizer stages its groups like the tiles");
constexpr int kColScaleGroups = 8;

struct ColItem {
    int64_t cw;          // first column of the item
    int64_t r_begin;     // first row
    int64_t r_end;       // one past the last row
    int64_t ngroups;
};

__device__ __forceinline__ ColItem col_item(int64_t it, int64_t gx, int64_t rows, int64_t rows_per_item) {
    ColItem ci;
    ci.cw = (it % gx) * kColCols;
    ci.r_begin = (it / gx) * rows_per_item;
    ci.r_end = min(rows, ci.r_begin + rows_per_item);
    ci.ngroups = (ci.r_end - ci.r_begin + kColGroupRB * 16 - 1) / (kColGroupRB * 16);
    return ci;
}

// SR of 16 rows x 4 columns (row pairs 2k, 2k+1 per conversion) into the
// column-wise payload words pk[j][0..1]; Philox words are made per row pair.
// A row pair with a flagged element (see sr_bucket) has its 8 nibbles redone
// in software.  get(j, r): value of row r, column j of the 16 x 4 block
// (compile-time indices after unrolling).
// S23: the values are formed scaled (x (r 2^23)) for the conversions and the
// bucket check; the software rounding takes x r.
template <bool ALIGNED, bool S23 = false, typename Get>
__device__ __forceinline__ void sr_cols16x4_v(Get get, const BlockScale (&bs)[4], uint64_t e_row0,
                                              uint64_t cols, uint32_t tid, uint32_t k0, uint32_t k1,
                                              uint32_t (&pk)[4][2]) {
    uint32_t aL[4][2] = {{0u, 0u}, {0u, 0u}, {0u, 0u}, {0u, 0u}};
    uint32_t aH[4][2] = {{0u, 0u}, {0u, 0u}, {0u, 0u}, {0u, 0u}};
    float ry[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) ry[j] = S23 ? bs[j].r * kS23 : bs[j].r;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        uint32_t n0[4], n1[4];
        nwords4<ALIGNED>(e_row0 + (uint64_t)(2 * k) * cols, tid, k0, k1, n0);
        nwords4<ALIGNED>(e_row0 + (uint64_t)(2 * k + 1) * cols, tid, k0, k1, n1);
        float y0[4], y1[4];
        uint32_t tb = 0u;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            y0[j] = get(j, 2 * k) * ry[j];
            y1[j] = get(j, 2 * k + 1) * ry[j];
            const v2f_t v = {y0[j], y1[j]};
            const uint32_t r1 = __builtin_amdgcn_alignbit(n1[j], n1[j], 1);
            uint32_t& L = aL[j][k >> 2];
            uint32_t& H = aH[j][k >> 2];
            if ((k & 3) == 0) { L = sr_pair<0, S23>(L, v, n0[j]); H = sr_pair<0, S23>(H, v, r1); }
            if ((k & 3) == 1) { L = sr_pair<1, S23>(L, v, n0[j]); H = sr_pair<1, S23>(H, v, r1); }
            if ((k & 3) == 2) { L = sr_pair<2, S23>(L, v, n0[j]); H = sr_pair<2, S23>(H, v, r1); }
            if ((k & 3) == 3) { L = sr_pair<3, S23>(L, v, n0[j]); H = sr_pair<3, S23>(H, v, r1); }
            tb = max(tb, max(sr_bucket<S23>(y0[j], n0[j]), sr_bucket<S23>(y1[j], n1[j])));
        }
        if (tb > kBucketTop) {
            const int sh = 8 * (k & 3);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                uint32_t& L = aL[j][k >> 2];
                uint32_t& H = aH[j][k >> 2];
                const float e0 = S23 ? get(j, 2 * k) * bs[j].r : y0[j];
                const float e1 = S23 ? get(j, 2 * k + 1) * bs[j].r : y1[j];
                L = (L & ~(0xFu << sh)) | (e2m1_sr(e0, ~n0[j]) << sh);
                H = (H & ~(0xF0u << sh)) | (e2m1_sr(e1, ~n1[j]) << (sh + 4));
            }
        }
        // one row pair at a time: keeps 8 Philox words live, not 64
        __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int h = 0; h < 2; ++h) pk[j][h] = (aL[j][h] & 0x0F0F0F0Fu) | (aH[j][h] & 0xF0F0F0F0u);
}

// The 16 x 4 block held as bf16 pairs: columns (c, c+1) in lo, (c+2, c+3) in hi.
template <bool ALIGNED, bool S23 = false>
__device__ __forceinline__ void sr_cols16x4(const uint32_t (&lo)[16], const uint32_t (&hi)[16],
                                            const BlockScale (&bs)[4], uint64_t e_row0, uint64_t cols,
                                            uint32_t tid, uint32_t k0, uint32_t k1,
                                            uint32_t (&pk)[4][2]) {
    sr_cols16x4_v<ALIGNED, S23>(
        [&](int j, int r) -> float {
            const uint32_t a = j < 2 ? lo[r] : hi[r];
            return (j & 1) ? bf16_hi(a) : bf16_lo(a);
        },
        bs, e_row0, cols, tid, k0, k1, pk);
}

// RHT: every 16-row block of each column is first replaced by its 16-point
// randomized Hadamard transform (rht16, sign mask rht_mask) and quantized as
// binary32 values (UE5M3 / E4M3 only).
template <bool SR, int FMT, bool RHT, int H>
__global__ __launch_bounds__(kThreads) void quant_cols_kernel(
    const uint16_t* __restrict__ x, int64_t rows, int64_t cols, int64_t rows_per_item, int64_t gx,
    int64_t nitems, const float* __restrict__ amax_dev, float T, uint32_t key0, uint32_t key1,
    uint32_t tid, uint8_t* __restrict__ payload_t, uint8_t* __restrict__ scales_t,
    float* __restrict__ dec_out, uint32_t rht_mask) {
    static_assert(!RHT || (FMT != (int)ScaleKind::E8M0 && H == 1), "transformed blocks are 16 rows");
    static_assert(FMT != (int)ScaleKind::E8M0 || H == 2, "E8M0 blocks are 32");
    __shared__ __attribute__((aligned(16))) uint8_t stP[kColGroupRB][kColCols * 8];
    __shared__ __attribute__((aligned(16))) uint8_t stS[kColCols][kColGroupRB * kColScaleGroups];
    __shared__ float rtab[256];
    // Blocks of 32 rows (H = 2): the two 16-row blocks of a wave (lanes l and
    // l + 32) form one block and share its maximum and scale byte.
    const Multipliers m = kernel_multipliers<FMT>(amax_dev, T);
    if (dec_out != nullptr && blockIdx.x == 0 && threadIdx.x == 0) *dec_out = m.dec;
    fill_recip<FMT>(rtab, m);
    const int t = threadIdx.x;
    const int q = t & 31, rbl = t >> 5;
    const bool vec8 = (cols & 3) == 0;
    const int64_t nrb = rows / (16 * H);                        // scale bytes per column
    const int64_t ldo = rows / 2;                               // payload_t row stride (bytes)

    // 16 rows x 4 columns of this lane's row block of group g of item ci:
    // word pairs (c, c+1) in lo, (c+2, c+3) in hi.
    auto load = [&](const ColItem& ci, int64_t g, uint32_t (&lo)[16], uint32_t (&hi)[16]) {
        const int64_t r0 = ci.r_begin + g * (kColGroupRB * 16) + rbl * 16;
        const int64_t c = ci.cw + 4 * q;
        const int64_t ncv = min((int64_t)4, cols - c);
        if (r0 >= ci.r_end || ncv <= 0) return;
        const uint16_t* src = x + r0 * cols + c;
        if (vec8 && ncv == 4) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const uint2 v = *reinterpret_cast<const uint2*>(src + r * cols);
                lo[r] = v.x;
                hi[r] = v.y;
            }
        } else {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                lo[r] = *reinterpret_cast<const uint32_t*>(src + r * cols);
                hi[r] = ncv == 4 ? *reinterpret_cast<const uint32_t*>(src + r * cols + 2) : 0u;
            }
        }
    };

    // S23: the scaled SR form (a uniform choice per launch, see kS23MaxG)
    auto run = [&](auto S23c) {
        constexpr bool S23 = decltype(S23c)::value;
        int64_t it = blockIdx.x, g = 0;
        if (it >= nitems) return;                                    // uniform
        ColItem ci = col_item(it, gx, rows, rows_per_item);
        uint32_t lo[16], hi[16], nlo[16], nhi[16];
        load(ci, 0, lo, hi);
        while (true) {
            // next group: within the item, else the first group of the next item
            int64_t nit = it, ng = g + 1;
            if (ng >= ci.ngroups) {
                nit = it + gridDim.x;
                ng = 0;
            }
            const ColItem cn = nit < nitems ? col_item(nit, gx, rows, rows_per_item) : ci;
            // RN prefetches the next group into registers; SR (VALU-bound)
            // keeps its registers for more resident waves and loads the next
            // group into the same registers once this one's values are consumed
            if (!SR && nit < nitems) load(cn, ng, nlo, nhi);

            const int64_t c = ci.cw + 4 * q;
            const int64_t r0 = ci.r_begin + g * (kColGroupRB * 16) + rbl * 16;
            const int sg = (int)(g % kColScaleGroups);
            if (RHT && r0 < ci.r_end && c < cols) {
                float v[4][16];
                BlockScale bs[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        v[j][r] = (j & 1) ? bf16_hi(j < 2 ? lo[r] : hi[r]) : bf16_lo(j < 2 ? lo[r] : hi[r]);
                    rht16(v[j], rht_mask);
                    uint32_t mb = 0u;
#pragma unroll
                    for (int r = 0; r < 16; ++r) mb = max(mb, __float_as_uint(v[j][r]) & 0x7FFFFFFFu);
                    bs[j] = block_scale_value<FMT>(__uint_as_float(mb), m, rtab);
                }
                uint32_t pk[4][2];
                if (SR) {
                    auto get = [&](int j, int r) -> float { return v[j][r]; };
                    if (vec8)
                        sr_cols16x4_v<true, S23>(get, bs, (uint64_t)r0 * (uint64_t)cols + (uint64_t)c, (uint64_t)cols,
                                            tid, key0, key1, pk);
                    else
                        sr_cols16x4_v<false, S23>(get, bs, (uint64_t)r0 * (uint64_t)cols + (uint64_t)c, (uint64_t)cols,
                                             tid, key0, key1, pk);
                } else {
                    const uint32_t nw[16] = {};
#pragma unroll
                    for (int j = 0; j < 4; ++j) quant_col16<false>(v[j], bs[j].r, nw, pk[j][0], pk[j][1]);
                }
                stage_cols4(stP[rbl], q, pk);
#pragma unroll
                for (int j = 0; j < 4; ++j) stS[4 * q + j][sg * kColGroupRB + rbl] = (uint8_t)bs[j].code;
            } else if (!RHT && r0 < ci.r_end && c < cols) {
                // packed 16-bit maxima of |x|: columns (c, c+1) and (c+2, c+3)
                uint32_t mL = 0u, mH = 0u;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    mL = pk_max_u16(mL, lo[r] & 0x7FFF7FFFu);
                    mH = pk_max_u16(mH, hi[r] & 0x7FFF7FFFu);
                }
                uint32_t mx[4] = {mL & 0xFFFFu, mL >> 16, mH & 0xFFFFu, mH >> 16};
                if (H == 2) {
#pragma unroll
                    for (int j = 0; j < 4; ++j) mx[j] = max(mx[j], (uint32_t)__shfl_xor((int)mx[j], 32));
                }
                BlockScale bs[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) bs[j] = block_scale<FMT>(mx[j], m, rtab);
                uint32_t pk[4][2];
                if (SR) {
                    if (vec8)
                        sr_cols16x4<true, S23>(lo, hi, bs, (uint64_t)r0 * (uint64_t)cols + (uint64_t)c,
                                          (uint64_t)cols, tid, key0, key1, pk);
                    else
                        sr_cols16x4<false, S23>(lo, hi, bs, (uint64_t)r0 * (uint64_t)cols + (uint64_t)c,
                                           (uint64_t)cols, tid, key0, key1, pk);
                } else {
                    const uint32_t nw[16] = {};
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        float xv[16];
#pragma unroll
                        for (int r = 0; r < 16; ++r)
                            xv[r] = (j & 1) ? bf16_hi(j < 2 ? lo[r] : hi[r]) : bf16_lo(j < 2 ? lo[r] : hi[r]);
                        quant_col16<false>(xv, bs[j].r, nw, pk[j][0], pk[j][1]);
                    }
                }
                stage_cols4(stP[rbl], q, pk);
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (H == 1 || (rbl & 1) == 0)
                        stS[4 * q + j][(sg * kColGroupRB + rbl) / H] = (uint8_t)bs[j].code;
            }
            // SR: this group's values are consumed; the next group's loads go out
            // now and overlap the stores below (same registers, none added)
            if (SR && nit < nitems) load(cn, ng, lo, hi);
            __syncthreads();
            // payload: 64-byte runs per column (the group's valid row
            // blocks only; a full group is 64 contiguous bytes)
            {
                const int col = t >> 1, half = t & 1;
                const int64_t gc = ci.cw + col;
                const int64_t rb0 = (ci.r_begin + g * (kColGroupRB * 16)) / 16;
                const int nvalid = (int)min((int64_t)kColGroupRB, (ci.r_end / 16) - rb0);
                store_cols64(stP, payload_t, ci.cw, cols, ldo, rb0 * 8, nvalid, t);
                // scales: at the end of the item (or of a full 64-block chunk);
                // SB bytes per column for a full chunk, half of them per lane
                if (sg == kColScaleGroups - 1 || g == ci.ngroups - 1) {
                    constexpr int SB = kColGroupRB * kColScaleGroups / H;
                    const int64_t rbs = (rb0 - (int64_t)sg * kColGroupRB) / H;
                    const int ns = (int)((rb0 + nvalid) / H - rbs);
                    if (gc < cols) {
                        uint8_t* dst = scales_t + gc * nrb + rbs + half * (SB / 2);
                        const uint8_t* s = &stS[col][half * (SB / 2)];
                        const int lo_k = half * (SB / 2), hi_k = min(ns, (half + 1) * (SB / 2));
                        if (hi_k - lo_k == SB / 2 && ((reinterpret_cast<uintptr_t>(dst) & 15) == 0)) {
#pragma unroll
                            for (int v = 0; v < SB / 32; ++v)
                                reinterpret_cast<uint4*>(dst)[v] = reinterpret_cast<const uint4*>(s)[v];
                        } else {
                            for (int k = lo_k; k < hi_k; ++k) dst[k - lo_k] = s[k - lo_k];
                        }
                    }
                }
            }
            __syncthreads();
            if (nit >= nitems) break;                               // uniform
            it = nit;
            g = ng;
            ci = cn;
            if (!SR) {
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    lo[r] = nlo[r];
                    hi[r] = nhi[r];
                }
            }
        }
    };
    if (SR && FMT != (int)ScaleKind::E8M0 && m.G <= kS23MaxG)
        run(std::integral_constant<bool, SR && FMT != (int)ScaleKind::E8M0>{});
    else
        run(std::false_type{});
}

// ------------------------------------------------------------ tiles (2D) --
// A workgroup covers 128 rows (8 tile rows; thread t handles tile row t / 32)
// x 128 columns (lane q = t % 32 holds columns 4q .. 4q+3, so the 4 lanes
// 4k .. 4k+3 share one 16x16 tile and combine their maxima with two lane
// swaps).  The row-major payload is stored straight from registers (32 lanes
// x 2 bytes = 64 contiguous bytes per row); the transposed payload gains 8
// bytes per tile row per column and is assembled in LDS, 64 bytes per column.

// TB: tile edge, 16 (the recipe) or 32 (the block-size control: a 32 x 32
// tile spans the 8 lanes of 32 columns and the lane pair l, l + 32 of two
// 16-row tile rows, all in one wave).
// Tile (column band bc, row band br) of walk index it on a gx x gy grid of
// 128 x 128 tiles.  Workgroups are dispatched round-robin over the 8 XCDs,
// so walk index it runs on XCD it % 8 (for a persistent walk: with a grid
// that is a multiple of 8).  With gx and gy multiples of 8 the tiles form
// 8 x 8 superblocks; XCD x takes superblocks x, x + 8, ... of the largest
// multiple of 8 of them, walked row by row, and the few superblocks left
// over follow in plain order.  Every 64-byte run of scale codes and every
// 128-byte line of transposed payload is then written by tiles of one XCD
// close together in time, so that XCD's L2 assembles whole lines before
// they are written back (8-byte pieces from different XCDs leave it as
// partial-line writes).  Otherwise row-major order.
__device__ __forceinline__ void xcd_tile(int64_t it, int64_t gx, int64_t gy, int64_t& bc, int64_t& br) {
    if ((gx & 7) != 0 || (gy & 7) != 0) {
        bc = it % gx;
        br = it / gx;
        return;
    }
    const int64_t nsb = (gx >> 3) * (gy >> 3);
    const int64_t even = (nsb & ~(int64_t)7) * 64;     // tiles of the superblocks dealt over the XCDs
    int64_t sbi, u;
    if (it < even) {
        const int64_t s = it >> 3;
        sbi = (it & 7) + 8 * (s >> 6);
        u = s & 63;
    } else {
        sbi = (nsb & ~(int64_t)7) + ((it - even) >> 6);
        u = (it - even) & 63;
    }
    bc = (sbi % (gx >> 3)) * 8 + (u & 7);
    br = (sbi / (gx >> 3)) * 8 + (u >> 3);
}

template <bool SR, int FMT, int TB = 16>
__global__ __launch_bounds__(kThreads) void quant_tiles_kernel(
    const uint16_t* __restrict__ w, int64_t rows, int64_t cols, const float* __restrict__ amax_dev,
    float T, uint32_t key0, uint32_t key1, uint32_t tid, uint8_t* __restrict__ payload,
    uint8_t* __restrict__ scales, uint8_t* __restrict__ payload_t, uint8_t* __restrict__ scales_t,
    float* __restrict__ dec_out) {
    __shared__ __attribute__((aligned(16))) uint8_t stT[kTileRowTiles][kTileCols * 8];
    __shared__ float rtab[256];
    static_assert(FMT != (int)ScaleKind::E8M0, "2D tiles take UE5M3 or E4M3 scales");
    const Multipliers m = kernel_multipliers<FMT>(amax_dev, T);
    if (dec_out != nullptr && blockIdx.x == 0 && threadIdx.x == 0) *dec_out = m.dec;
    fill_recip<FMT>(rtab, m);
    const int t = threadIdx.x;
    const int q = t & 31, trl = t >> 5;
    int64_t bc, br;
    xcd_tile(blockIdx.x, (cols + kTileCols - 1) / kTileCols, (rows / 16 + kTileRowTiles - 1) / kTileRowTiles, bc,
             br);
    const int64_t cw = bc * kTileCols;
    const int64_t c = cw + 4 * q;
    const int64_t tr = br * kTileRowTiles + trl;                      // tile row
    const int64_t ntr = rows / 16, ntc = cols / 16;
    const bool active = (c < cols) && (tr < ntr);                     // whole tiles: cols % 16 == 0
    if (active) {
        const uint16_t* src = w + (tr * 16) * cols + c;
        uint32_t lo[16], hi[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const uint2 v = *reinterpret_cast<const uint2*>(src + r * cols);
            lo[r] = v.x;
            hi[r] = v.y;
        }
        uint32_t mx = 0;
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = max(mx, max(bf16_abs_max_pair(lo[r]), bf16_abs_max_pair(hi[r])));
        mx = max(mx, (uint32_t)__shfl_xor((int)mx, 1));
        mx = max(mx, (uint32_t)__shfl_xor((int)mx, 2));
        if (TB == 32) {
            mx = max(mx, (uint32_t)__shfl_xor((int)mx, 4));
            mx = max(mx, (uint32_t)__shfl_xor((int)mx, 32));
        }
        const BlockScale bs = block_scale<FMT>(mx, m, rtab);
        uint32_t colpk[4][2] = {{0u, 0u}, {0u, 0u}, {0u, 0u}, {0u, 0u}};
        if (SR) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                uint32_t wd[4];
                words4((uint64_t)(tr * 16 + r) * (uint64_t)cols + (uint64_t)c, tid, key0, key1, wd);
                const float xv[4] = {bf16_lo(lo[r]), bf16_hi(lo[r]), bf16_lo(hi[r]), bf16_hi(hi[r])};
                uint32_t p = 0;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const uint32_t nib = e2m1_sr(xv[j] * bs.r, wd[j]);
                    p |= nib << (4 * j);
                    colpk[j][r >> 3] |= nib << (4 * (r & 7));
                }
                *reinterpret_cast<uint16_t*>(payload + (tr * 16 + r) * (cols / 2) + c / 2) = (uint16_t)p;
            }
        } else {
            // row-major pairs (columns c, c+1 and c+2, c+3) and, for the
            // transposed payload, column-wise pairs of consecutive rows
            float y[16][4];
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                y[r][0] = bf16_lo(lo[r]) * bs.r;
                y[r][1] = bf16_hi(lo[r]) * bs.r;
                y[r][2] = bf16_lo(hi[r]) * bs.r;
                y[r][3] = bf16_hi(hi[r]) * bs.r;
                uint32_t p = 0;
                p = rn_pair<0>(p, y[r][0], y[r][1]);
                p = rn_pair<1>(p, y[r][2], y[r][3]);
                *reinterpret_cast<uint16_t*>(payload + (tr * 16 + r) * (cols / 2) + c / 2) = (uint16_t)p;
            }
            if (payload_t != nullptr) {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    uint32_t a = 0u, b = 0u;
                    a = rn_pair<0>(a, y[0][j], y[1][j]);
                    a = rn_pair<1>(a, y[2][j], y[3][j]);
                    a = rn_pair<2>(a, y[4][j], y[5][j]);
                    a = rn_pair<3>(a, y[6][j], y[7][j]);
                    b = rn_pair<0>(b, y[8][j], y[9][j]);
                    b = rn_pair<1>(b, y[10][j], y[11][j]);
                    b = rn_pair<2>(b, y[12][j], y[13][j]);
                    b = rn_pair<3>(b, y[14][j], y[15][j]);
                    colpk[j][0] = a;
                    colpk[j][1] = b;
                }
            }
        }
        if (TB == 16 && (q & 3) == 0) {
            scales[tr * ntc + c / 16] = (uint8_t)bs.code;
            if (scales_t != nullptr) scales_t[(c / 16) * ntr + tr] = (uint8_t)bs.code;
        }
        if (TB == 32 && (q & 7) == 0 && (trl & 1) == 0) {
            scales[(tr / 2) * (ntc / 2) + c / 32] = (uint8_t)bs.code;
            if (scales_t != nullptr) scales_t[(c / 32) * (ntr / 2) + tr / 2] = (uint8_t)bs.code;
        }
        if (payload_t != nullptr) {
            stage_cols4(stT[trl], q, colpk);
        }
    }
    if (payload_t == nullptr) return;                                 // uniform
    __syncthreads();
    store_cols64(stT, payload_t, cw, cols, rows / 2, br * kTileRowTiles * 8,
                 (int)min((int64_t)kTileRowTiles, ntr - br * kTileRowTiles), t);
}

// ------------------------------------------------- both axes in one pass --
// The row blocking (blocks of 16 along each row) and the column blocking
// (blocks of 16 down each column, stored transposed) of one tensor from a
// single read of it -- the two operands of a backward pass (dY: dgrad and
// wgrad) or of X (fprop and wgrad).  A tile is 128 rows (8 tile rows; thread
// t handles tile row t / 32) x 128 columns (lane q = t % 32 holds columns
// 4q .. 4q+3), i.e. a 16 x 4 piece per lane: its 4 column blocks are
// in-lane, each row block spans the 4 lanes 4k .. 4k+3 (maxima combined by
// two quad permutations).  Row payloads go out straight from registers (32
// lanes x 2 bytes = 64 contiguous bytes per row); the transposed payload and
// both scale arrays are assembled in LDS.  SR words use tensor id tid_r for
// the row blocking and tid_c for the column blocking.
//
// Persistent: workgroup w walks tiles w, w + grid, ... (tile columns
// fastest), loading the next tile while it quantizes the current one.  The
// LDS stage alternates between two buffers, so one barrier per tile
// separates a tile's LDS writes from its stores and the stores of tile k
// from the writes of tile k + 2.

// The RN work of one lane's 16 x 4 piece of a dual-axis tile: lo / hi hold
// rows r of columns (c, c+1) / (c+2, c+3) as bf16 pairs.  Writes the
// transposed column payload (4 columns x 8 bytes) and the column scale codes
// to the LDS stage, the row scale codes of the rows this lane owns in its
// quad, and the row payload (2 bytes per row) to prow (row stride rstride
// bytes).  Per element: its 15-bit |x| enters packed 16-bit maxima shared by
// the two blockings, and its binary32 value is formed once and multiplied by
// the row and the column reciprocal (the same binary32 products as the
// single-axis quantizers).
template <int FMT>
__device__ __forceinline__ void dual_rn_tile(const uint32_t (&lo)[16], const uint32_t (&hi)[16],
                                             const Multipliers& m, const float* rtab,
                                             uint8_t (*P)[kTileCols * 8],
                                             uint8_t (*SC)[kTileRowTiles], uint8_t (*SRo)[kTileCols / 16],
                                             int q, int trl, uint8_t* __restrict__ prow, int64_t rstride) {
    uint32_t mcL = 0u, mcH = 0u;              // packed column maxima: (c, c+1), (c+2, c+3)
    uint32_t mrow[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const uint32_t a = lo[r] & 0x7FFF7FFFu, b = hi[r] & 0x7FFF7FFFu;
        mcL = pk_max_u16(mcL, a);
        mcH = pk_max_u16(mcH, b);
        const uint32_t ab = pk_max_u16(a, b);
        uint32_t mr = max(ab & 0xFFFFu, ab >> 16);
        mr = max(mr, (uint32_t)__builtin_amdgcn_mov_dpp((int)mr, 0xB1, 0xF, 0xF, false));   // quad xor 1
        mr = max(mr, (uint32_t)__builtin_amdgcn_mov_dpp((int)mr, 0x4E, 0xF, 0xF, false));   // quad xor 2
        mrow[r] = mr;
    }
    BlockScale bc[4];
    bc[0] = block_scale<FMT>(mcL & 0xFFFFu, m, rtab);
    bc[1] = block_scale<FMT>(mcL >> 16, m, rtab);
    bc[2] = block_scale<FMT>(mcH & 0xFFFFu, m, rtab);
    bc[3] = block_scale<FMT>(mcH >> 16, m, rtab);
    // lane k of the quad derives the scales of rows k, k+4, k+8, k+12; the
    // others take them by a quad broadcast
    const int qk = q & 3;
    BlockScale own[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const uint32_t mo = qk == 0 ? mrow[4 * u] : qk == 1 ? mrow[4 * u + 1] : qk == 2 ? mrow[4 * u + 2] : mrow[4 * u + 3];
        own[u] = block_scale<FMT>(mo, m, rtab);
        SRo[trl * 16 + 4 * u + qk][q >> 2] = (uint8_t)own[u].code;
    }
    uint32_t cp[4][2] = {{0u, 0u}, {0u, 0u}, {0u, 0u}, {0u, 0u}};
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        float xv[2][4];
        float rr[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int r = 2 * k + h;
            xv[h][0] = bf16_lo(lo[r]);
            xv[h][1] = bf16_hi(lo[r]);
            xv[h][2] = bf16_lo(hi[r]);
            xv[h][3] = bf16_hi(hi[r]);
            const int ov = __float_as_int(own[r >> 2].r);
            const int src = r & 3;
            rr[h] = __int_as_float(src == 0 ? __builtin_amdgcn_mov_dpp(ov, 0x00, 0xF, 0xF, false)
                                   : src == 1 ? __builtin_amdgcn_mov_dpp(ov, 0x55, 0xF, 0xF, false)
                                   : src == 2 ? __builtin_amdgcn_mov_dpp(ov, 0xAA, 0xF, 0xF, false)
                                              : __builtin_amdgcn_mov_dpp(ov, 0xFF, 0xF, 0xF, false));
            uint32_t p = 0u;
            p = rn_pair<0>(p, xv[h][0] * rr[h], xv[h][1] * rr[h]);
            p = rn_pair<1>(p, xv[h][2] * rr[h], xv[h][3] * rr[h]);
            *reinterpret_cast<uint16_t*>(prow + r * rstride) = (uint16_t)p;
        }
        // columns: rows 2k, 2k+1 of each column form one nibble pair
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            uint32_t& w = cp[j][k >> 2];
            const float y0 = xv[0][j] * bc[j].r, y1 = xv[1][j] * bc[j].r;
            if ((k & 3) == 0) w = rn_pair<0>(w, y0, y1);
            if ((k & 3) == 1) w = rn_pair<1>(w, y0, y1);
            if ((k & 3) == 2) w = rn_pair<2>(w, y0, y1);
            if ((k & 3) == 3) w = rn_pair<3>(w, y0, y1);
        }
    }
    stage_cols4(P[trl], q, cp);
#pragma unroll
    for (int j = 0; j < 4; ++j) SC[4 * q + j][trl] = (uint8_t)bc[j].code;
}

struct DualStage {
    uint8_t P[kTileRowTiles][kTileCols * 8];          // transposed payload (see store_cols64)
    uint8_t SR[kTileRowTiles * 16][kTileCols / 16];   // row scales, 8 per row
    uint8_t SC[kTileCols][kTileRowTiles];             // column scales, 8 per column
};

template <bool SR, int FMT>
__global__ __launch_bounds__(kThreads) void quant_dual_kernel(
    const uint16_t* __restrict__ x, int64_t rows, int64_t cols, int64_t gx, int64_t ntiles,
    const float* __restrict__ amax_dev, float T, uint32_t key0, uint32_t key1, uint32_t tid_r,
    uint32_t tid_c, uint8_t* __restrict__ payload_r, uint8_t* __restrict__ scales_r,
    uint8_t* __restrict__ payload_c, uint8_t* __restrict__ scales_c, float* __restrict__ dec_out) {
    __shared__ __attribute__((aligned(16))) DualStage stage[2];
    __shared__ float rtab[256];
    static_assert(FMT != (int)ScaleKind::E8M0, "blocks of 16");
    const Multipliers m = kernel_multipliers<FMT>(amax_dev, T);
    if (dec_out != nullptr && blockIdx.x == 0 && threadIdx.x == 0) *dec_out = m.dec;
    fill_recip<FMT>(rtab, m);
    const int t = threadIdx.x;
    const int q = t & 31, trl = t >> 5;
    const int64_t ntr = rows / 16;
    const bool vec_scales = (cols % 128) == 0 && (ntr % 8) == 0;   // 8-byte scale runs aligned
    const int64_t gy = ntiles / gx;

    // 16 rows x 4 columns of this lane's piece of tile `it`: word pairs
    // (c, c+1) in L, (c+2, c+3) in H (left untouched outside the tensor).
    // The input is read once: non-temporal loads keep it from displacing
    // the partly written output lines in L2.
    auto load = [&](int64_t it, uint32_t (&L)[16], uint32_t (&H)[16]) {
        int64_t bc, br;
        xcd_tile(it, gx, gy, bc, br);
        const int64_t c = bc * kTileCols + 4 * q;
        const int64_t tr = br * kTileRowTiles + trl;
        if (c >= cols || tr >= ntr) return;                           // cols % 16 == 0: whole pieces
        const uint16_t* src = x + (tr * 16) * cols + c;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const u32x2_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x2_t*>(src + r * cols));
            L[r] = v.x;
            H[r] = v.y;
        }
    };

    int64_t it = blockIdx.x;
    if (it >= ntiles) return;                                        // uniform
    // RN prefetches the next tile into registers; SR (VALU-bound: Philox for
    // both blockings) keeps its registers for more resident waves instead
    constexpr bool kPrefetch = !SR;
    uint32_t lo[16], hi[16], nlo[16], nhi[16];
    load(it, lo, hi);
    for (int buf = 0;; buf ^= 1) {
        const int64_t nit = it + gridDim.x;
        if (kPrefetch && nit < ntiles) load(nit, nlo, nhi);
        DualStage& st = stage[buf];
        int64_t bcol, brow;
        xcd_tile(it, gx, gy, bcol, brow);
        const int64_t cw = bcol * kTileCols;
        const int64_t c = cw + 4 * q;
        const int64_t tr0 = brow * kTileRowTiles;
        const int64_t tr = tr0 + trl;
        if (!SR && c < cols && tr < ntr) {
            // RN: block maxima from the |x| bits, both blockings' scales, then
            // one pass over row pairs that widens each element once for its
            // row and its column conversion
            dual_rn_tile<FMT>(lo, hi, m, rtab, st.P, st.SC, st.SR, q, trl,
                              payload_r + (tr * 16) * (cols / 2) + c / 2, cols / 2);
        } else if (SR && c < cols && tr < ntr) {
            // column blocks: in-lane maxima of the 4 columns
            uint32_t mL = 0u, mH = 0u;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                mL = pk_max_u16(mL, lo[r] & 0x7FFF7FFFu);
                mH = pk_max_u16(mH, hi[r] & 0x7FFF7FFFu);
            }
            const uint32_t mc[4] = {mL & 0xFFFFu, mL >> 16, mH & 0xFFFFu, mH >> 16};
            BlockScale bc[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) bc[j] = block_scale<FMT>(mc[j], m, rtab);
            uint32_t pk[4][2];
            if (SR) {
                sr_cols16x4<true>(lo, hi, bc, (uint64_t)(tr * 16) * (uint64_t)cols + (uint64_t)c,
                                  (uint64_t)cols, tid_c, key0, key1, pk);
            } else {
                const uint32_t nw[16] = {};
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    float xv[16];
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        xv[r] = (j & 1) ? bf16_hi(j < 2 ? lo[r] : hi[r]) : bf16_lo(j < 2 ? lo[r] : hi[r]);
                    quant_col16<false>(xv, bc[j].r, nw, pk[j][0], pk[j][1]);
                }
            }
            stage_cols4(st.P[trl], q, pk);
#pragma unroll
            for (int j = 0; j < 4; ++j) st.SC[4 * q + j][trl] = (uint8_t)bc[j].code;
            // row blocks: one per row over the lane quad 4k .. 4k+3.  Maxima
            // are combined by quad permutations; lane k of the quad derives
            // the scales of rows k, k+4, k+8, k+12 and the others take them
            // by a quad broadcast, so each block scale is computed once.
            uint32_t mrow[16];
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                uint32_t mr = max(bf16_abs_max_pair(lo[r]), bf16_abs_max_pair(hi[r]));
                mr = max(mr, (uint32_t)__builtin_amdgcn_mov_dpp((int)mr, 0xB1, 0xF, 0xF, false));   // quad xor 1
                mr = max(mr, (uint32_t)__builtin_amdgcn_mov_dpp((int)mr, 0x4E, 0xF, 0xF, false));   // quad xor 2
                mrow[r] = mr;
            }
            const int qk = q & 3;
            BlockScale own[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                // row 4u + qk of this lane's quad position
                const uint32_t mo = qk == 0 ? mrow[4 * u] : qk == 1 ? mrow[4 * u + 1]
                                  : qk == 2 ? mrow[4 * u + 2] : mrow[4 * u + 3];
                own[u] = block_scale<FMT>(mo, m, rtab);
            }
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                // broadcast of quad lane r % 4 (its own[r / 4])
                BlockScale br;
                const int ov = __float_as_int(own[r >> 2].r);
                const int src = r & 3;
                br.r = __int_as_float(src == 0 ? __builtin_amdgcn_mov_dpp(ov, 0x00, 0xF, 0xF, false)
                                      : src == 1 ? __builtin_amdgcn_mov_dpp(ov, 0x55, 0xF, 0xF, false)
                                      : src == 2 ? __builtin_amdgcn_mov_dpp(ov, 0xAA, 0xF, 0xF, false)
                                                 : __builtin_amdgcn_mov_dpp(ov, 0xFF, 0xF, 0xF, false));
                br.code = own[r >> 2].code;              // valid in quad lane r % 4, which stores it
                const float y[4] = {bf16_lo(lo[r]) * br.r, bf16_hi(lo[r]) * br.r, bf16_lo(hi[r]) * br.r,
                                    bf16_hi(hi[r]) * br.r};
                uint32_t p;
                if (SR) {
                    uint32_t nw[4];
                    nwords4<true>((uint64_t)(tr * 16 + r) * (uint64_t)cols + (uint64_t)c, tid_r, key0, key1, nw);
                    p = sr4(y, nw);
                } else {
                    p = 0u;
                    p = rn_pair<0>(p, y[0], y[1]);
                    p = rn_pair<1>(p, y[2], y[3]);
                }
                *reinterpret_cast<uint16_t*>(payload_r + (tr * 16 + r) * (cols / 2) + c / 2) = (uint16_t)p;
                if (qk == (r & 3)) st.SR[trl * 16 + r][q >> 2] = (uint8_t)br.code;
                // one row at a time: keeps the live Philox words to 4
                if (SR) __builtin_amdgcn_sched_barrier(0);
            }
        }
        __syncthreads();
        const int nvalid = (int)min((int64_t)kTileRowTiles, ntr - tr0);
        // transposed payload: 64-byte runs per column
        store_cols64(st.P, payload_c, cw, cols, rows / 2, tr0 * 8, nvalid, t);
        if (t < kTileCols) {
            // column scales [cols, rows/16]: 8 bytes per column
            const int64_t gc = cw + t;
            if (gc < cols) {
                uint8_t* dst = scales_c + gc * ntr + tr0;
                if (vec_scales && nvalid == kTileRowTiles)
                    *reinterpret_cast<uint2*>(dst) = *reinterpret_cast<const uint2*>(&st.SC[t][0]);
                else
                    for (int k = 0; k < nvalid; ++k) dst[k] = st.SC[t][k];
            }
        } else {
            // row scales [rows, cols/16]: 8 bytes per row
            const int row = t - kTileCols;
            const int64_t gr = tr0 * 16 + row;
            if (row < nvalid * 16) {
                const int64_t nb = min((int64_t)(kTileCols / 16), (cols - cw) / 16);
                uint8_t* dst = scales_r + gr * (cols / 16) + cw / 16;
                if (vec_scales && nb == kTileCols / 16)
                    *reinterpret_cast<uint2*>(dst) = *reinterpret_cast<const uint2*>(&st.SR[row][0]);
                else
                    for (int k = 0; k < nb; ++k) dst[k] = st.SR[row][k];
            }
        }
        if (nit >= ntiles) break;                                   // uniform
        it = nit;
        if (kPrefetch) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                lo[r] = nlo[r];
                hi[r] = nhi[r];
            }
        } else {
            load(it, lo, hi);
        }
    }
}

inline void seed_key(uint64_t seed, uint32_t& k0, uint32_t& k1) {
    k0 = (uint32_t)seed;
    k1 = (uint32_t)(seed >> 32);
}

// Resident workgroups to aim for: 8 per CU on the 256 CUs of an MI355X.
constexpr int64_t kPersistentWGs = 256 * 8;

template <int FMT, int H>
hipError_t launch_rows_fmt(const void* x_bf16, int64_t rows, int64_t cols, const float* amax_dev,
                           float target, bool sr, uint64_t seed, uint32_t tensor_id,
                           uint8_t* payload, uint8_t* scales, float* dec_out, hipStream_t s) {
    constexpr int64_t BE = 16 * H;
    const int64_t nblocks = rows * cols / BE;
    uint32_t k0, k1;
    seed_key(seed, k0, k1);
    int64_t wgs = (nblocks + kThreads - 1) / kThreads;
    if (wgs < 1) wgs = 1;
    if (wgs > kPersistentWGs) wgs = kPersistentWGs;
    const uint4* x = reinterpret_cast<const uint4*>(x_bf16);
    uint2* p = reinterpret_cast<uint2*>(payload);
    if (sr)
        hipLaunchKernelGGL((quant_rows_kernel<true, FMT, H>), dim3((unsigned)wgs), dim3(kThreads), 0, s, x,
                           nblocks, amax_dev, target, k0, k1, tensor_id, p, scales, dec_out);
    else
        hipLaunchKernelGGL((quant_rows_kernel<false, FMT, H>), dim3((unsigned)wgs), dim3(kThreads), 0, s, x,
                           nblocks, amax_dev, target, k0, k1, tensor_id, p, scales, dec_out);
    return hipGetLastError();
}

// Resident workgroups of a kernel on the current device (cached per device;
// threads that race here store the same value).
template <typename K>
int64_t resident_wgs(K kernel, int slot) {
    static std::atomic<int64_t> cache[16][16];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 16) return kPersistentWGs;
    int64_t v = cache[dev][slot].load(std::memory_order_relaxed);
    if (v == 0) {
        int cus = 0, per = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, reinterpret_cast<const void*>(kernel),
                                                         kThreads, 0) != hipSuccess ||
            cus <= 0 || per <= 0)
            return kPersistentWGs;
        v = (int64_t)cus * per;
        cache[dev][slot].store(v, std::memory_order_relaxed);
    }
    return v;
}

template <int FMT, int H, bool RHT = false>
hipError_t launch_cols_fmt(const void* x_bf16, int64_t rows, int64_t cols, const float* amax_dev,
                           float target, bool sr, uint64_t seed, uint32_t tensor_id,
                           uint8_t* payload_t, uint8_t* scales_t, float* dec_out, hipStream_t s,
                           uint32_t rht_mask = 0u) {
    uint32_t k0, k1;
    seed_key(seed, k0, k1);
    const int64_t gx = (cols + kColCols - 1) / kColCols;
    const int slot = 2 * FMT + (RHT ? 6 : 0) + (H == 2 && FMT != (int)ScaleKind::E8M0 ? 8 : 0);
    const int64_t resident = sr ? resident_wgs(quant_cols_kernel<true, FMT, RHT, H>, slot)
                                : resident_wgs(quant_cols_kernel<false, FMT, RHT, H>, slot + 1);
    // Items of up to 64 row blocks (whole 64-byte scale runs); shorter when
    // that leaves fewer than 2 items per resident workgroup.
    int64_t rows_per_item = (int64_t)kColGroupRB * kColScaleGroups * 16;     // 1024 rows
    while (rows_per_item > kColGroupRB * 16 &&
           gx * ((rows + rows_per_item - 1) / rows_per_item) < 2 * resident)
        rows_per_item /= 2;
    const int64_t nitems = gx * ((rows + rows_per_item - 1) / rows_per_item);
    const int64_t grid = min(nitems, resident);
    const uint16_t* x = reinterpret_cast<const uint16_t*>(x_bf16);
    if (sr)
        hipLaunchKernelGGL((quant_cols_kernel<true, FMT, RHT, H>), dim3((unsigned)grid), dim3(kThreads), 0, s, x,
                           rows, cols, rows_per_item, gx, nitems, amax_dev, target, k0, k1, tensor_id,
                           payload_t, scales_t, dec_out, rht_mask);
    else
        hipLaunchKernelGGL((quant_cols_kernel<false, FMT, RHT, H>), dim3((unsigned)grid), dim3(kThreads), 0, s, x,
                           rows, cols, rows_per_item, gx, nitems, amax_dev, target, k0, k1, tensor_id,
                           payload_t, scales_t, dec_out, rht_mask);
    return hipGetLastError();
}

template <int FMT, int TB>
hipError_t launch_tiles_fmt(const void* w_bf16, int64_t rows, int64_t cols, const float* amax_dev,
                            float target, bool sr, uint64_t seed, uint32_t tensor_id,
                            uint8_t* payload, uint8_t* scales, uint8_t* payload_t, uint8_t* scales_t,
                            float* dec_out, hipStream_t s) {
    uint32_t k0, k1;
    seed_key(seed, k0, k1);
    const int64_t gx = (cols + kTileCols - 1) / kTileCols;
    const int64_t gy = (rows / 16 + kTileRowTiles - 1) / kTileRowTiles;
    const uint16_t* w = reinterpret_cast<const uint16_t*>(w_bf16);
    if (sr)
        hipLaunchKernelGGL((quant_tiles_kernel<true, FMT, TB>), dim3((unsigned)(gx * gy)), dim3(kThreads),
                           0, s, w, rows, cols, amax_dev, target, k0, k1, tensor_id, payload, scales,
                           payload_t, scales_t, dec_out);
    else
        hipLaunchKernelGGL((quant_tiles_kernel<false, FMT, TB>), dim3((unsigned)(gx * gy)), dim3(kThreads),
                           0, s, w, rows, cols, amax_dev, target, k0, k1, tensor_id, payload, scales,
                           payload_t, scales_t, dec_out);
    return hipGetLastError();
}

template <int FMT>
hipError_t launch_dual_fmt(const void* x_bf16, int64_t rows, int64_t cols, const float* amax_dev,
                           float target, bool sr, uint64_t seed, uint32_t tid_r, uint32_t tid_c,
                           uint8_t* payload_r, uint8_t* scales_r, uint8_t* payload_c, uint8_t* scales_c,
                           float* dec_out, hipStream_t s) {
    uint32_t k0, k1;
    seed_key(seed, k0, k1);
    const int64_t gx = (cols + kTileCols - 1) / kTileCols;
    const int64_t gy = (rows / 16 + kTileRowTiles - 1) / kTileRowTiles;
    const int64_t ntiles = gx * gy;
    const int64_t resident = sr ? resident_wgs(quant_dual_kernel<true, FMT>, 12 + FMT)
                                : resident_wgs(quant_dual_kernel<false, FMT>, 14 + FMT);
    // SR: one tile per workgroup (measured faster than the persistent walk
    // for the VALU-bound SR form); RN: persistent, next tile prefetched
    const int64_t grid = sr ? ntiles : min(ntiles, resident);
    const uint16_t* x = reinterpret_cast<const uint16_t*>(x_bf16);
    if (sr)
        hipLaunchKernelGGL((quant_dual_kernel<true, FMT>), dim3((unsigned)grid), dim3(kThreads), 0, s, x, rows,
                           cols, gx, ntiles, amax_dev, target, k0, k1, tid_r, tid_c, payload_r, scales_r,
                           payload_c, scales_c, dec_out);
    else
        hipLaunchKernelGGL((quant_dual_kernel<false, FMT>), dim3((unsigned)grid), dim3(kThreads), 0, s, x, rows,
                           cols, gx, ntiles, amax_dev, target, k0, k1, tid_r, tid_c, payload_r, scales_r,
                           payload_c, scales_c, dec_out);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_quant_rows(ScaleKind fmt, int block, const void* x_bf16, int64_t rows, int64_t cols,
                             const float* amax_dev, float target, bool sr, uint64_t seed,
                             uint32_t tensor_id, uint8_t* payload, uint8_t* scales,
                             float* dec_out, hipStream_t s) {
#define UE5M3_ROWS(F, H) launch_rows_fmt<(int)ScaleKind::F, H>(x_bf16, rows, cols, amax_dev, target, sr, seed, \
                                                              tensor_id, payload, scales, dec_out, s)
    switch (fmt) {
        case ScaleKind::E4M3: return block == 32 ? UE5M3_ROWS(E4M3, 2) : UE5M3_ROWS(E4M3, 1);
        case ScaleKind::E8M0: return UE5M3_ROWS(E8M0, 2);
        default: return block == 32 ? UE5M3_ROWS(UE5M3, 2) : UE5M3_ROWS(UE5M3, 1);
    }
#undef UE5M3_ROWS
}

hipError_t launch_quant_cols(ScaleKind fmt, int block, const void* x_bf16, int64_t rows, int64_t cols,
                             const float* amax_dev, float target, bool sr, uint64_t seed,
                             uint32_t tensor_id, uint8_t* payload_t, uint8_t* scales_t,
                             float* dec_out, hipStream_t s) {
#define UE5M3_COLS(F, H) launch_cols_fmt<(int)ScaleKind::F, H>(x_bf16, rows, cols, amax_dev, target, sr, seed, \
                                                              tensor_id, payload_t, scales_t, dec_out, s)
    switch (fmt) {
        case ScaleKind::E4M3: return block == 32 ? UE5M3_COLS(E4M3, 2) : UE5M3_COLS(E4M3, 1);
        case ScaleKind::E8M0: return UE5M3_COLS(E8M0, 2);
        default: return block == 32 ? UE5M3_COLS(UE5M3, 2) : UE5M3_COLS(UE5M3, 1);
    }
#undef UE5M3_COLS
}

hipError_t launch_quant_cols_rht(const void* x_bf16, int64_t rows, int64_t cols, const float* amax_dev,
                                 float target, bool sr, uint64_t seed, uint32_t tensor_id,
                                 uint32_t sign_mask, uint8_t* payload_t, uint8_t* scales_t,
                                 float* dec_out, hipStream_t s) {
    return launch_cols_fmt<(int)ScaleKind::UE5M3, 1, true>(x_bf16, rows, cols, amax_dev, target, sr, seed,
                                                        tensor_id, payload_t, scales_t, dec_out, s,
                                                        sign_mask);
}

hipError_t launch_quant_tiles(ScaleKind fmt, int tile, const void* w_bf16, int64_t rows, int64_t cols,
                              const float* amax_dev, float target, bool sr, uint64_t seed,
                              uint32_t tensor_id, uint8_t* payload, uint8_t* scales,
                              uint8_t* payload_t, uint8_t* scales_t, float* dec_out,
                              hipStream_t s) {
#define UE5M3_TILES(F, TB) launch_tiles_fmt<(int)ScaleKind::F, TB>(w_bf16, rows, cols, amax_dev, target, sr, \
                               seed, tensor_id, payload, scales, payload_t, scales_t, dec_out, s)
    if (fmt == ScaleKind::E4M3) return tile == 32 ? UE5M3_TILES(E4M3, 32) : UE5M3_TILES(E4M3, 16);
    return tile == 32 ? UE5M3_TILES(UE5M3, 32) : UE5M3_TILES(UE5M3, 16);
#undef UE5M3_TILES
}

hipError_t launch_quant_dual(ScaleKind fmt, const void* x_bf16, int64_t rows, int64_t cols,
                             const float* amax_dev, float target, bool sr, uint64_t seed,
                             uint32_t tid_r, uint32_t tid_c, uint8_t* payload_r, uint8_t* scales_r,
                             uint8_t* payload_c, uint8_t* scales_c, float* dec_out, hipStream_t s) {
    if (fmt == ScaleKind::E4M3)
        return launch_dual_fmt<(int)ScaleKind::E4M3>(x_bf16, rows, cols, amax_dev, target, sr, seed, tid_r,
                                                     tid_c, payload_r, scales_r, payload_c, scales_c,
                                                     dec_out, s);
    return launch_dual_fmt<(int)ScaleKind::UE5M3>(x_bf16, rows, cols, amax_dev, target, sr, seed, tid_r,
                                                  tid_c, payload_r, scales_r, payload_c, scales_c, dec_out,
                                                  s);
}

}  // namespace ue5m3
