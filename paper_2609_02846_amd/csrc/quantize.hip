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
// bytes for the optional transposed weight payload.
#include "codec.hpp"
#include "launch.hpp"

namespace ue5m3 {
namespace {

constexpr int kThreads = 256;

struct BlockScale {
    uint32_t code;
    float r;
};

__device__ __forceinline__ BlockScale block_scale(uint32_t amax_bits15, const Multipliers& m) {
    const float a = __uint_as_float(amax_bits15 << 16);
    uint32_t code = ue5m3_encode(a * m.S);
    code = code ? code : kCodeOne;
    BlockScale bs;
    bs.code = code;
    bs.r = m.G / ue5m3_decode(code);
    return bs;
}

// Quantize the 8 bf16 values held in v (element e in half e&1 of word e>>1)
// with reciprocal r; returns 8 nibbles packed little-endian.  For SR, w holds
// the 8 Philox words of the elements.
template <bool SR>
__device__ __forceinline__ uint32_t quant8(const uint32_t (&v)[4], float r, const uint32_t* w) {
    uint32_t p = 0;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const float x = (e & 1) ? bf16_hi(v[e >> 1]) : bf16_lo(v[e >> 1]);
        const float y = x * r;
        const uint32_t nib = SR ? e2m1_sr(y, w[e]) : e2m1_rn(y);
        p |= nib << (4 * e);
    }
    return p;
}

__device__ __forceinline__ void words8(uint64_t first_elem, uint32_t tid, uint32_t k0, uint32_t k1,
                                       uint32_t* w) {
    // first_elem is a multiple of 4: two Philox blocks cover the 8 elements
    const uint4 a = sr_words4(first_elem >> 2, tid, k0, k1);
    const uint4 b = sr_words4((first_elem >> 2) + 1, tid, k0, k1);
    w[0] = a.x; w[1] = a.y; w[2] = a.z; w[3] = a.w;
    w[4] = b.x; w[5] = b.y; w[6] = b.z; w[7] = b.w;
}

// ------------------------------------------------------------ rows (1D) --
// The flat tensor is a sequence of 16-element blocks (cols % 16 == 0).  Each
// lane handles one 8-element chunk (16 B); lanes 2k, 2k+1 hold one block and
// combine their maxima with a lane swap.  Payload: 4 B per chunk, scale: 1 B
// per block written by the even lane.
constexpr int kRowUnroll = 4;

template <bool SR>
__global__ __launch_bounds__(kThreads) void quant_rows_kernel(
    const uint4* __restrict__ x, int64_t nchunks, const float* __restrict__ amax_dev, float T,
    uint32_t key0, uint32_t key1, uint32_t tid, uint32_t* __restrict__ payload,
    uint8_t* __restrict__ scales, float* __restrict__ dec_out) {
    const Multipliers m = tensor_multipliers(*amax_dev, T);
    if (dec_out != nullptr && blockIdx.x == 0 && threadIdx.x == 0) *dec_out = m.dec;
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    for (int64_t base = (int64_t)blockIdx.x * kThreads + threadIdx.x; base < nchunks;
         base += stride * kRowUnroll) {
        uint4 v[kRowUnroll];
#pragma unroll
        for (int u = 0; u < kRowUnroll; ++u) {
            const int64_t c = base + u * stride;
            if (c < nchunks) v[u] = x[c];
        }
#pragma unroll
        for (int u = 0; u < kRowUnroll; ++u) {
            const int64_t c = base + u * stride;
            if (c < nchunks) {   // uniform within each lane pair (nchunks is even)
                const uint32_t vv[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
                uint32_t mx = max(max(bf16_abs_max_pair(vv[0]), bf16_abs_max_pair(vv[1])),
                                  max(bf16_abs_max_pair(vv[2]), bf16_abs_max_pair(vv[3])));
                mx = max(mx, (uint32_t)__shfl_xor((int)mx, 1));
                const BlockScale bs = block_scale(mx, m);
                uint32_t w[8];
                if (SR) words8((uint64_t)c * 8, tid, key0, key1, w);
                payload[c] = quant8<SR>(vv, bs.r, w);
                if ((c & 1) == 0) scales[c >> 1] = (uint8_t)bs.code;
            }
        }
    }
}

// ------------------------------------------------ columns (1D, transposed) --
// Blocks are 16 consecutive rows of one column; output is the row blocking of
// x^T.  A lane holds 4 adjacent columns (8 B per row) of kColRB consecutive
// row blocks; a workgroup covers 256 columns x (4 waves * kColRB * 16) rows,
// so each output row (a column of x) receives 4 * kColRB * 8 contiguous
// payload bytes from one workgroup.
constexpr int kColRB = 4;
constexpr int kColWaves = kThreads / 64;

template <bool SR>
__global__ __launch_bounds__(kThreads) void quant_cols_kernel(
    const uint16_t* __restrict__ x, int64_t rows, int64_t cols, const float* __restrict__ amax_dev,
    float T, uint32_t key0, uint32_t key1, uint32_t tid, uint8_t* __restrict__ payload_t,
    uint8_t* __restrict__ scales_t, float* __restrict__ dec_out) {
    const Multipliers m = tensor_multipliers(*amax_dev, T);
    if (dec_out != nullptr && blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) *dec_out = m.dec;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int64_t c0 = ((int64_t)blockIdx.x * 64 + lane) * 4;     // first of 4 columns
    if (c0 >= cols) return;
    const bool pair2 = (c0 + 2) < cols;                            // columns c0+2, c0+3 exist
    const bool vec8 = (cols & 3) == 0;                             // 8-byte aligned rows
    const int64_t nrb = rows / 16;
    const int64_t rb_first = ((int64_t)blockIdx.y * kColWaves + wave) * kColRB;
    const int64_t ldo = rows / 2;        // payload_t row stride (bytes)
#pragma unroll 1
    for (int q = 0; q < kColRB; ++q) {
        const int64_t rb = rb_first + q;
        if (rb >= nrb) break;
        uint32_t lo[16], hi[16];         // bf16 pairs: columns (c0, c0+1), (c0+2, c0+3)
        const uint16_t* src = x + (rb * 16) * cols + c0;
        if (pair2 && vec8) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const uint2 t = *reinterpret_cast<const uint2*>(src + r * cols);
                lo[r] = t.x;
                hi[r] = t.y;
            }
        } else {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                lo[r] = *reinterpret_cast<const uint32_t*>(src + r * cols);
                hi[r] = pair2 ? *reinterpret_cast<const uint32_t*>(src + r * cols + 2) : 0u;
            }
        }
        // column maxima (integer on |bf16| bits)
        uint32_t mx[4] = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            mx[0] = max(mx[0], lo[r] & 0x7FFFu);
            mx[1] = max(mx[1], (lo[r] >> 16) & 0x7FFFu);
            mx[2] = max(mx[2], hi[r] & 0x7FFFu);
            mx[3] = max(mx[3], (hi[r] >> 16) & 0x7FFFu);
        }
        BlockScale bs[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) bs[j] = block_scale(mx[j], m);
        uint32_t pk[4][2] = {{0u, 0u}, {0u, 0u}, {0u, 0u}, {0u, 0u}};
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            float xv[4] = {bf16_lo(lo[r]), bf16_hi(lo[r]), bf16_lo(hi[r]), bf16_hi(hi[r])};
            uint32_t w[4] = {0u, 0u, 0u, 0u};
            if (SR) {
                // elements (row, c0 .. c0+3); c0 % 4 == 0 and cols % 4 == 0 put
                // them in one Philox block, otherwise they straddle two.
                const uint64_t e0 = (uint64_t)(rb * 16 + r) * (uint64_t)cols + (uint64_t)c0;
                const uint4 wa = sr_words4(e0 >> 2, tid, key0, key1);
                if ((e0 & 3) == 0) {
                    w[0] = wa.x; w[1] = wa.y; w[2] = wa.z; w[3] = wa.w;
                } else {         // e0 is even: the 4 elements straddle two blocks
                    const uint4 wb = sr_words4((e0 >> 2) + 1, tid, key0, key1);
                    w[0] = wa.z; w[1] = wa.w; w[2] = wb.x; w[3] = wb.y;
                }
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const float y = xv[j] * bs[j].r;
                const uint32_t nib = SR ? e2m1_sr(y, w[j]) : e2m1_rn(y);
                pk[j][r >> 3] |= nib << (4 * (r & 7));
            }
        }
        const int ncol = pair2 ? 4 : 2;
        for (int j = 0; j < ncol; ++j) {
            uint8_t* dst = payload_t + (c0 + j) * ldo + rb * 8;
            *reinterpret_cast<uint2*>(dst) = make_uint2(pk[j][0], pk[j][1]);
            scales_t[(c0 + j) * nrb + rb] = (uint8_t)bs[j].code;
        }
    }
}

// ------------------------------------------------------------ tiles (2D) --
// A lane holds 16 rows x 8 columns (16 B per row); lanes 2k, 2k+1 cover one
// 16x16 tile and combine their maxima with a lane swap.  A workgroup covers
// 512 columns x (4 waves * kTileRT * 16) rows.
constexpr int kTileRT = 2;

template <bool SR>
__global__ __launch_bounds__(kThreads) void quant_tiles_kernel(
    const uint16_t* __restrict__ w, int64_t rows, int64_t cols, const float* __restrict__ amax_dev,
    float T, uint32_t key0, uint32_t key1, uint32_t tid, uint8_t* __restrict__ payload,
    uint8_t* __restrict__ scales, uint8_t* __restrict__ payload_t, uint8_t* __restrict__ scales_t,
    float* __restrict__ dec_out) {
    const Multipliers m = tensor_multipliers(*amax_dev, T);
    if (dec_out != nullptr && blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) *dec_out = m.dec;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int64_t c0 = ((int64_t)blockIdx.x * 64 + lane) * 8;
    if (c0 >= cols) return;              // cols % 16 == 0: lane pairs leave together
    const int64_t ntr = rows / 16, ntc = cols / 16;
    const int64_t tr_first = ((int64_t)blockIdx.y * kColWaves + wave) * kTileRT;
#pragma unroll 1
    for (int q = 0; q < kTileRT; ++q) {
        const int64_t tr = tr_first + q;
        if (tr >= ntr) break;            // uniform within the wave
        uint4 v[16];
        const uint16_t* src = w + (tr * 16) * cols + c0;
#pragma unroll
        for (int r = 0; r < 16; ++r) v[r] = *reinterpret_cast<const uint4*>(src + r * cols);
        uint32_t mx = 0;
#pragma unroll
        for (int r = 0; r < 16; ++r)
            mx = max(mx, max(max(bf16_abs_max_pair(v[r].x), bf16_abs_max_pair(v[r].y)),
                             max(bf16_abs_max_pair(v[r].z), bf16_abs_max_pair(v[r].w))));
        mx = max(mx, (uint32_t)__shfl_xor((int)mx, 1));
        const BlockScale bs = block_scale(mx, m);
        uint32_t colpk[8][2];
#pragma unroll
        for (int j = 0; j < 8; ++j) colpk[j][0] = colpk[j][1] = 0u;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const uint32_t vv[4] = {v[r].x, v[r].y, v[r].z, v[r].w};
            uint32_t wd[8];
            if (SR) words8((uint64_t)(tr * 16 + r) * (uint64_t)cols + (uint64_t)c0, tid, key0, key1, wd);
            const uint32_t p = quant8<SR>(vv, bs.r, wd);
            *reinterpret_cast<uint32_t*>(payload + (tr * 16 + r) * (cols / 2) + c0 / 2) = p;
#pragma unroll
            for (int j = 0; j < 8; ++j) colpk[j][r >> 3] |= ((p >> (4 * j)) & 15u) << (4 * (r & 7));
        }
        if ((lane & 1) == 0) {
            scales[tr * ntc + c0 / 16] = (uint8_t)bs.code;
            if (scales_t != nullptr) scales_t[(c0 / 16) * ntr + tr] = (uint8_t)bs.code;
        }
        if (payload_t != nullptr) {
#pragma unroll
            for (int j = 0; j < 8; ++j)
                *reinterpret_cast<uint2*>(payload_t + (c0 + j) * (rows / 2) + tr * 8) =
                    make_uint2(colpk[j][0], colpk[j][1]);
        }
    }
}

inline void seed_key(uint64_t seed, uint32_t& k0, uint32_t& k1) {
    k0 = (uint32_t)seed;
    k1 = (uint32_t)(seed >> 32);
}

}  // namespace

hipError_t launch_quant_rows(const void* x_bf16, int64_t rows, int64_t cols,
                             const float* amax_dev, float target, bool sr, uint64_t seed,
                             uint32_t tensor_id, uint8_t* payload, uint8_t* scales,
                             float* dec_out, hipStream_t s) {
    const int64_t nchunks = rows * cols / 8;
    uint32_t k0, k1;
    seed_key(seed, k0, k1);
    int64_t blocks = (nchunks + (int64_t)kThreads * kRowUnroll - 1) / ((int64_t)kThreads * kRowUnroll);
    if (blocks < 1) blocks = 1;
    if (blocks > 8192) blocks = 8192;
    const uint4* x = reinterpret_cast<const uint4*>(x_bf16);
    uint32_t* p = reinterpret_cast<uint32_t*>(payload);
    if (sr)
        hipLaunchKernelGGL(quant_rows_kernel<true>, dim3((unsigned)blocks), dim3(kThreads), 0, s, x,
                           nchunks, amax_dev, target, k0, k1, tensor_id, p, scales, dec_out);
    else
        hipLaunchKernelGGL(quant_rows_kernel<false>, dim3((unsigned)blocks), dim3(kThreads), 0, s, x,
                           nchunks, amax_dev, target, k0, k1, tensor_id, p, scales, dec_out);
    return hipGetLastError();
}

hipError_t launch_quant_cols(const void* x_bf16, int64_t rows, int64_t cols,
                             const float* amax_dev, float target, bool sr, uint64_t seed,
                             uint32_t tensor_id, uint8_t* payload_t, uint8_t* scales_t,
                             float* dec_out, hipStream_t s) {
    uint32_t k0, k1;
    seed_key(seed, k0, k1);
    const int64_t gx = (cols + 255) / 256;
    const int64_t rows_per_wg = (int64_t)kColWaves * kColRB * 16;
    int64_t gy = (rows + rows_per_wg - 1) / rows_per_wg;
    if (gy < 1) gy = 1;
    const uint16_t* x = reinterpret_cast<const uint16_t*>(x_bf16);
    if (sr)
        hipLaunchKernelGGL(quant_cols_kernel<true>, dim3((unsigned)gx, (unsigned)gy), dim3(kThreads),
                           0, s, x, rows, cols, amax_dev, target, k0, k1, tensor_id, payload_t,
                           scales_t, dec_out);
    else
        hipLaunchKernelGGL(quant_cols_kernel<false>, dim3((unsigned)gx, (unsigned)gy), dim3(kThreads),
                           0, s, x, rows, cols, amax_dev, target, k0, k1, tensor_id, payload_t,
                           scales_t, dec_out);
    return hipGetLastError();
}

hipError_t launch_quant_tiles(const void* w_bf16, int64_t rows, int64_t cols,
                              const float* amax_dev, float target, bool sr, uint64_t seed,
                              uint32_t tensor_id, uint8_t* payload, uint8_t* scales,
                              uint8_t* payload_t, uint8_t* scales_t, float* dec_out,
                              hipStream_t s) {
    uint32_t k0, k1;
    seed_key(seed, k0, k1);
    const int64_t gx = (cols + 511) / 512;
    const int64_t rows_per_wg = (int64_t)kColWaves * kTileRT * 16;
    const int64_t gy = (rows + rows_per_wg - 1) / rows_per_wg;
    const uint16_t* w = reinterpret_cast<const uint16_t*>(w_bf16);
    if (sr)
        hipLaunchKernelGGL(quant_tiles_kernel<true>, dim3((unsigned)gx, (unsigned)gy), dim3(kThreads),
                           0, s, w, rows, cols, amax_dev, target, k0, k1, tensor_id, payload, scales,
                           payload_t, scales_t, dec_out);
    else
        hipLaunchKernelGGL(quant_tiles_kernel<false>, dim3((unsigned)gx, (unsigned)gy), dim3(kThreads),
                           0, s, w, rows, cols, amax_dev, target, k0, k1, tensor_id, payload, scales,
                           payload_t, scales_t, dec_out);
    return hipGetLastError();
}

}  // namespace ue5m3
