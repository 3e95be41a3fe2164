// 16-point randomized Hadamard transform of one column block, used on the
// weight-gradient operands (the "UE5M3 with Transformer Engine settings"
// recipe, paper Table 6 and Sec. 2): y = (1/4) H16 diag(s) x with H16 the
// Sylvester Hadamard matrix (H[i][j] = (-1)^popcount(i & j)) and s_i = -1
// where bit i of the sign mask is set.  Binary32 evaluation order: sign
// flips (exact), butterfly stages h = 1, 2, 4, 8 -- (u_i, u_{i+h}) <-
// (u_i + u_{i+h}, u_i - u_{i+h}) for every i with bit h clear, one rounding
// each -- then the exact scaling by 1/4.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ue5m3 {

__device__ __forceinline__ void rht16(float (&u)[16], uint32_t mask) {
#pragma unroll
    for (int i = 0; i < 16; ++i) u[i] = __uint_as_float(__float_as_uint(u[i]) ^ (((mask >> i) & 1u) << 31));
#pragma unroll
    for (int h = 1; h < 16; h <<= 1) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            if ((i & h) == 0) {
                const float a = u[i], b = u[i + h];
                u[i] = a + b;
                u[i + h] = a - b;
            }
        }
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) u[i] *= 0.25f;
}

}  // namespace ue5m3
