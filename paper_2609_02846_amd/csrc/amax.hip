// Tensor amax of a bf16 tensor (paper Sec. 4.1: a_t = max_i |x_{t,i}|),
// launched only on refresh steps of the sample-and-hold rule, or without the
// clear as a running maximum over calibration batches (the calibrated-frozen
// inference reference).
//
// The maximum is exact: |x| of a bf16 is its 15 low bits, and the integer
// order of those bits is the numeric order of non-negative finite values, so
// the kernel takes an integer max and stores the binary32 bits of the result
// (bf16 bits << 16).  HBM-bound streaming read, 2 bytes per element.
#include "codec.hpp"
#include "launch.hpp"
#include "rht.hpp"

namespace ue5m3 {
namespace {

constexpr int kAmaxThreads = 256;
constexpr int kAmaxUnroll = 4;

__global__ void amax_clear_kernel(uint32_t* out) {
    if (threadIdx.x == 0) out[0] = 0u;
}

__global__ __launch_bounds__(kAmaxThreads) void amax_bf16_kernel(
    const uint4* __restrict__ x16, int64_t nvec, const uint16_t* __restrict__ tail,
    int tail_n, uint32_t* __restrict__ out) {
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
    // wavefront reduction, then one atomic per workgroup
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off));
    __shared__ uint32_t red[kAmaxThreads / 64];
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) red[wave] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t r = red[0];
        for (int w = 1; w < kAmaxThreads / 64; ++w) r = max(r, red[w]);
        atomicMax(out, r << 16);
    }
}

// Amax of the transformed tensor: item i covers 16 rows (block i / npairs)
// of two adjacent columns (pair i % npairs), so consecutive lanes read
// consecutive 4-byte pairs of a row.  rows % 16 == 0, cols % 2 == 0.
__global__ __launch_bounds__(kAmaxThreads) void amax_rht_kernel(
    const uint16_t* __restrict__ x, int64_t rows, int64_t cols, uint32_t mask, uint32_t* __restrict__ out) {
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
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off));
    __shared__ uint32_t red[kAmaxThreads / 64];
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) red[wave] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t r = red[0];
        for (int w = 1; w < kAmaxThreads / 64; ++w) r = max(r, red[w]);
        atomicMax(out, r);
    }
}

}  // namespace

hipError_t launch_amax_rht(const void* x_bf16, int64_t rows, int64_t cols, uint32_t sign_mask,
                           float* amax_dev, hipStream_t s) {
    uint32_t* out = reinterpret_cast<uint32_t*>(amax_dev);
    hipLaunchKernelGGL(amax_clear_kernel, dim3(1), dim3(64), 0, s, out);
    const int64_t nitems = (rows / 16) * (cols / 2);
    if (nitems <= 0) return hipGetLastError();
    int64_t blocks = (nitems + kAmaxThreads - 1) / kAmaxThreads;
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(amax_rht_kernel, dim3((unsigned)blocks), dim3(kAmaxThreads), 0, s,
                       reinterpret_cast<const uint16_t*>(x_bf16), rows, cols, sign_mask, out);
    return hipGetLastError();
}

hipError_t launch_amax(const void* x_bf16, int64_t numel, float* amax_dev, bool clear,
                       hipStream_t s) {
    uint32_t* out = reinterpret_cast<uint32_t*>(amax_dev);
    if (clear) hipLaunchKernelGGL(amax_clear_kernel, dim3(1), dim3(64), 0, s, out);
    if (numel <= 0) return hipGetLastError();
    const int64_t nvec = numel / 8;
    const int tail_n = (int)(numel - nvec * 8);
    const uint16_t* tail = reinterpret_cast<const uint16_t*>(x_bf16) + nvec * 8;
    int64_t blocks = (nvec + kAmaxThreads * kAmaxUnroll - 1) / (kAmaxThreads * kAmaxUnroll);
    if (blocks < 1) blocks = 1;
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(amax_bf16_kernel, dim3((unsigned)blocks), dim3(kAmaxThreads), 0, s,
                       reinterpret_cast<const uint4*>(x_bf16), nvec, tail, tail_n, out);
    return hipGetLastError();
}

}  // namespace ue5m3
