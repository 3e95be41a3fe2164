// Tensor amax of a bf16 tensor (paper Sec. 4.1: a_t = max_i |x_{t,i}|),
// launched only on refresh steps of the sample-and-hold rule, or without the
// clear as a running maximum over calibration batches (the calibrated-frozen
// inference reference).
//
// The maximum is exact: |x| of a bf16 is its 15 low bits, and the integer
// order of those bits is the numeric order of non-negative finite values, so
// the kernel takes an integer max and stores the binary32 bits of the result
// (bf16 bits << 16).  HBM-bound streaming read, 2 bytes per element.
//
// Two launches and no atomics: each workgroup stores its maximum in a
// library workspace (one per device and stream), and one workgroup then
// reduces those partial maxima into *amax_dev.  (Thousands of device-scope
// atomics on one address serialize: with one atomic per workgroup the 64 MiB
// activation took ~60 us instead of ~15.)
#include "codec.hpp"
#include "launch.hpp"
#include "rht.hpp"

namespace ue5m3 {
namespace {

constexpr int kAmaxThreads = 256;
constexpr int kAmaxUnroll = 4;

constexpr int kAmaxMaxBlocks = 4096;

// out = max(keep ? out : 0, max of part[0 .. n) << shift) as binary32 bits.
__global__ __launch_bounds__(kAmaxThreads) void amax_final_kernel(const uint32_t* __restrict__ part, int n,
                                                                  int shift, int keep, uint32_t* __restrict__ out) {
    uint32_t m = 0;
    for (int i = threadIdx.x; i < n; i += kAmaxThreads) m = max(m, part[i]);
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off));
    __shared__ uint32_t red[kAmaxThreads / 64];
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) red[wave] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t r = red[0];
        for (int w = 1; w < kAmaxThreads / 64; ++w) r = max(r, red[w]);
        r <<= shift;
        out[0] = keep ? max(out[0], r) : r;
    }
}

// Workgroup maximum of m into part[blockIdx.x].
__device__ __forceinline__ void store_block_max(uint32_t m, uint32_t* __restrict__ part) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off));
    __shared__ uint32_t red[kAmaxThreads / 64];
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) red[wave] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t r = red[0];
        for (int w = 1; w < kAmaxThreads / 64; ++w) r = max(r, red[w]);
        part[blockIdx.x] = r;
    }
}

__global__ __launch_bounds__(kAmaxThreads) void amax_bf16_kernel(
    const uint4* __restrict__ x16, int64_t nvec, const uint16_t* __restrict__ tail,
    int tail_n, uint32_t* __restrict__ part) {
    uint32_t m = 0;
    const int64_t stride = (int64_t)gridDim.x * kAmaxThreads;
    int64_t i = (int64_t)blockIdx.x * kAmaxThreads + threadIdx.x;
    for (; i + (kAmaxUnroll - 1) * stride < nvec; i += kAmaxUnroll * stride) {
        uint4 v[kAmaxUnroll];
#pragma unroll
        for (int u = 0; u < kAmaxUnroll; ++u) v[u] = x16[i + u * stride];
#pragma unroll
        for (int u = 0; u < kAmaxUnroll; ++u) {
            m = max(m, bf16_abs_max_pair(v[u].x));
            m = max(m, bf16_abs_max_pair(v[u].y));
            m = max(m, bf16_abs_max_pair(v[u].z));
            m = max(m, bf16_abs_max_pair(v[u].w));
        }
    }
    for (; i < nvec; i += stride) {
        const uint4 v = x16[i];
        m = max(m, max(max(bf16_abs_max_pair(v.x), bf16_abs_max_pair(v.y)),
                       max(bf16_abs_max_pair(v.z), bf16_abs_max_pair(v.w))));
    }
    if (blockIdx.x == 0 && (int)threadIdx.x < tail_n) m = max(m, (uint32_t)(tail[threadIdx.x] & 0x7FFFu));
    store_block_max(m, part);
}

// Amax of the transformed tensor: item i covers 16 rows (block i / npairs)
// of two adjacent columns (pair i % npairs), so consecutive lanes read
// consecutive 4-byte pairs of a row.  rows % 16 == 0, cols % 2 == 0.
__global__ __launch_bounds__(kAmaxThreads) void amax_rht_kernel(
    const uint16_t* __restrict__ x, int64_t rows, int64_t cols, uint32_t mask, uint32_t* __restrict__ part) {
    const int64_t npairs = cols / 2;
    const int64_t nitems = (rows / 16) * npairs;
    uint32_t m = 0;
    for (int64_t i = (int64_t)blockIdx.x * kAmaxThreads + threadIdx.x; i < nitems;
         i += (int64_t)gridDim.x * kAmaxThreads) {
        const int64_t rb = i / npairs, cp = i - rb * npairs;
        const uint32_t* src = reinterpret_cast<const uint32_t*>(x + rb * 16 * cols + 2 * cp);
        float a[16], b[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const uint32_t w = src[r * (cols / 2)];
            a[r] = __uint_as_float(w << 16);
            b[r] = __uint_as_float(w & 0xFFFF0000u);
        }
        rht16(a, mask);
        rht16(b, mask);
#pragma unroll
        for (int r = 0; r < 16; ++r)
            m = max(m, max(__float_as_uint(a[r]) & 0x7FFFFFFFu, __float_as_uint(b[r]) & 0x7FFFFFFFu));
    }
    store_block_max(m, part);
}

// Partial maxima of `blocks` workgroups into the stream's workspace, then
// the final reduction (shift: 16 for bf16 magnitude bits, 0 for binary32).
template <typename Launch>
hipError_t amax_two_pass(int64_t blocks, int shift, bool keep, float* amax_dev, hipStream_t s, Launch launch) {
    uint32_t* out = reinterpret_cast<uint32_t*>(amax_dev);
    void* ws = nullptr;
    hipError_t e = stream_workspace(kWsAmax, s, kAmaxMaxBlocks * sizeof(uint32_t), &ws);
    if (e != hipSuccess) return e;
    uint32_t* part = static_cast<uint32_t*>(ws);
    if (blocks > 0) {
        launch(part);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    hipLaunchKernelGGL(amax_final_kernel, dim3(1), dim3(kAmaxThreads), 0, s, part, (int)blocks, shift,
                       keep ? 1 : 0, out);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_amax_rht(const void* x_bf16, int64_t rows, int64_t cols, uint32_t sign_mask,
                           float* amax_dev, hipStream_t s) {
    const int64_t nitems = (rows / 16) * (cols / 2);
    int64_t blocks = nitems <= 0 ? 0 : (nitems + kAmaxThreads - 1) / kAmaxThreads;
    if (blocks > kAmaxMaxBlocks) blocks = kAmaxMaxBlocks;
    return amax_two_pass(blocks, 0, false, amax_dev, s, [&](uint32_t* part) {
        hipLaunchKernelGGL(amax_rht_kernel, dim3((unsigned)blocks), dim3(kAmaxThreads), 0, s,
                           reinterpret_cast<const uint16_t*>(x_bf16), rows, cols, sign_mask, part);
    });
}

hipError_t launch_amax(const void* x_bf16, int64_t numel, float* amax_dev, bool clear,
                       hipStream_t s) {
    if (numel <= 0 && !clear) return hipSuccess;
    const int64_t nvec = numel > 0 ? numel / 8 : 0;
    const int tail_n = numel > 0 ? (int)(numel - nvec * 8) : 0;
    const uint16_t* tail = reinterpret_cast<const uint16_t*>(x_bf16) + nvec * 8;
    int64_t blocks = numel <= 0 ? 0 : (nvec + kAmaxThreads * kAmaxUnroll - 1) / (kAmaxThreads * kAmaxUnroll);
    if (numel > 0 && blocks < 1) blocks = 1;
    if (blocks > kAmaxMaxBlocks) blocks = kAmaxMaxBlocks;
    return amax_two_pass(blocks, 16, !clear, amax_dev, s, [&](uint32_t* part) {
        hipLaunchKernelGGL(amax_bf16_kernel, dim3((unsigned)blocks), dim3(kAmaxThreads), 0, s,
                           reinterpret_cast<const uint4*>(x_bf16), nvec, tail, tail_n, part);
    });
}

}  // namespace ue5m3
