// Internal launchers shared between the kernel sources and the C ABI shim.
// Each returns hipSuccess or the launch error; arguments are validated by the
// caller (api.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ue5m3 {

// B scale layouts: one code per (row, 16 k) or per (16 rows, 16 k).  TileDgrad
// is Tile for the dgrad product: the same code, instantiated separately so
// that profiles tell the fprop and dgrad launches apart.
enum class BScale : int { Row = 0, Tile = 1, TileDgrad = 2 };

hipError_t launch_amax(const void* x_bf16, int64_t numel, float* amax_dev, hipStream_t s);

hipError_t launch_quant_rows(const void* x_bf16, int64_t rows, int64_t cols,
                             const float* amax_dev, float target, bool sr, uint64_t seed,
                             uint32_t tensor_id, uint8_t* payload, uint8_t* scales,
                             float* dec_out, hipStream_t s);

hipError_t launch_quant_cols(const void* x_bf16, int64_t rows, int64_t cols,
                             const float* amax_dev, float target, bool sr, uint64_t seed,
                             uint32_t tensor_id, uint8_t* payload_t, uint8_t* scales_t,
                             float* dec_out, hipStream_t s);

hipError_t launch_quant_tiles(const void* w_bf16, int64_t rows, int64_t cols,
                              const float* amax_dev, float target, bool sr, uint64_t seed,
                              uint32_t tensor_id, uint8_t* payload, uint8_t* scales,
                              uint8_t* payload_t, uint8_t* scales_t, float* dec_out,
                              hipStream_t s);

hipError_t launch_gemm(BScale bmode, int64_t M, int64_t N, int64_t K,
                       const uint8_t* a, const uint8_t* a_scales, const float* a_dec,
                       const uint8_t* b, const uint8_t* b_scales, const float* b_dec,
                       void* c, bool c_bf16, hipStream_t s);

}  // namespace ue5m3
