// C ABI shim: argument validation, status mapping and dispatch to the kernel
// launchers.  See include/ue5m3.h for the contract of every entry point.
#include <cmath>
#include <cstdint>

#include "../../include/ue5m3.h"
#include "launch.hpp"

namespace {

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
inline bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

inline ue5m3_status_t hip_status(hipError_t e) { return e == hipSuccess ? UE5M3_OK : UE5M3_EHIP; }

inline bool valid_target(float t) { return std::isfinite(t) && t > 0.0f && std::isfinite(t * 6.0f); }

// Orientation of an operand blocking: blocks along the source's rows, down
// its columns (stored transposed), or square tiles.
enum class Orient { Row, ColT, Tile };

inline bool blocking_of(ue5m3_blocking_t b, int& len, Orient& o) {
    switch (b) {
        case UE5M3_ROW16: len = 16; o = Orient::Row; return true;
        case UE5M3_COL16T: len = 16; o = Orient::ColT; return true;
        case UE5M3_TILE16: len = 16; o = Orient::Tile; return true;
        case UE5M3_ROW32: len = 32; o = Orient::Row; return true;
        case UE5M3_COL32T: len = 32; o = Orient::ColT; return true;
        case UE5M3_TILE32: len = 32; o = Orient::Tile; return true;
    }
    return false;
}

// A blocking serves an operand whose source is contracted along its rows
// (rows_contracted) or down its columns when its blocks run along that
// contraction (eq:microscaling; Sec. 4.3): Row or Tile for the first, ColT
// or Tile for the second.
inline bool along_contraction(Orient o, bool rows_contracted) {
    return o == Orient::Tile || (o == Orient::Row) == rows_contracted;
}

// Operand checks shared by the GEMM entry points: the layout, the two
// blockings (valid values, equal block lengths, A one-dimensional, both
// along the contraction) and the B scale layout they select.  On success
// *block is the common block length.
ue5m3_status_t gemm_blockings(ue5m3_layout_t layout, ue5m3_blocking_t a_blk, ue5m3_blocking_t b_blk,
                              bool e8, int* block, ue5m3::BScale* bmode) {
    bool a_rows, b_rows;     // is the source contracted along its rows?
    switch (layout) {
        case UE5M3_NT: a_rows = true; b_rows = true; break;
        case UE5M3_NN: a_rows = true; b_rows = false; break;
        case UE5M3_TN: a_rows = false; b_rows = false; break;
        default: return UE5M3_ELAYOUT;
    }
    int la = 0, lb = 0;
    Orient oa = Orient::Row, ob = Orient::Row;
    if (!blocking_of(a_blk, la, oa) || !blocking_of(b_blk, lb, ob) || la != lb) return UE5M3_EINVAL;
    if (e8 && (la != 32 || oa == Orient::Tile || ob == Orient::Tile)) return UE5M3_EINVAL;
    if (oa == Orient::Tile || !along_contraction(oa, a_rows) || !along_contraction(ob, b_rows))
        return UE5M3_ELAYOUT;
    *block = la;
    if (ob != Orient::Tile)
        *bmode = ue5m3::BScale::Row;
    else
        *bmode = layout == UE5M3_NN ? ue5m3::BScale::TileDgrad : ue5m3::BScale::Tile;
    return UE5M3_OK;
}

}  // namespace

extern "C" {

int32_t ue5m3_version(void) { return 200; }

const char* ue5m3_status_string(ue5m3_status_t s) {
    switch (s) {
        case UE5M3_OK: return "ok";
        case UE5M3_EINVAL: return "invalid argument (null pointer, enum, target or period)";
        case UE5M3_ESHAPE: return "invalid shape (negative, or not a required multiple)";
        case UE5M3_EALIGN: return "pointer not 16-byte aligned";
        case UE5M3_ELAYOUT: return "unknown GEMM layout, or an operand blocking not along the contraction";
        case UE5M3_EHIP: return "HIP runtime or launch error";
        case UE5M3_ESCRATCH: return "the call needs more scratch than the allocation-free entry point holds";
    }
    return "unknown status";
}

ue5m3_status_t ue5m3_amax_state_init(ue5m3_amax_state_t* st, float* amax_dev, int32_t period) {
    if (st == nullptr || amax_dev == nullptr || period < 0) return UE5M3_EINVAL;
    if (!aligned4(amax_dev)) return UE5M3_EALIGN;
    st->amax_dev = amax_dev;
    st->last_refresh = 0;
    st->period = period;
    st->has_cache = 0;
    return UE5M3_OK;
}

void ue5m3_amax_state_reset(ue5m3_amax_state_t* st) {
    if (st != nullptr) {
        st->has_cache = 0;
        st->last_refresh = 0;
    }
}

ue5m3_status_t ue5m3_amax_sample(ue5m3_amax_state_t* st, const void* x_bf16, int64_t numel,
                                 int64_t step, int32_t* refreshed, hipStream_t stream) {
    if (st == nullptr || st->amax_dev == nullptr || st->period < 0) return UE5M3_EINVAL;
    if (numel < 0) return UE5M3_ESHAPE;
    if (numel > 0 && x_bf16 == nullptr) return UE5M3_EINVAL;
    if (numel > 0 && !aligned16(x_bf16)) return UE5M3_EALIGN;
    if (!aligned4(st->amax_dev)) return UE5M3_EALIGN;
    const bool refresh = !st->has_cache ||
                         (st->period > 0 && step - st->last_refresh >= (int64_t)st->period);
    if (refreshed != nullptr) *refreshed = refresh ? 1 : 0;
    if (!refresh) return UE5M3_OK;
    const hipError_t e = ue5m3::launch_amax(x_bf16, numel, st->amax_dev, true, stream);
    if (e != hipSuccess) return UE5M3_EHIP;
    st->has_cache = 1;
    st->last_refresh = step;
    return UE5M3_OK;
}

void ue5m3_amax_state_freeze(ue5m3_amax_state_t* st) {
    if (st != nullptr) {
        st->has_cache = 1;
        st->period = 0;
    }
}

ue5m3_status_t ue5m3_amax_accumulate(const void* x_bf16, int64_t numel, float* amax_dev,
                                     int32_t clear, hipStream_t stream) {
    if (amax_dev == nullptr || (clear != 0 && clear != 1)) return UE5M3_EINVAL;
    if (numel < 0) return UE5M3_ESHAPE;
    if (numel > 0 && x_bf16 == nullptr) return UE5M3_EINVAL;
    if (numel > 0 && !aligned16(x_bf16)) return UE5M3_EALIGN;
    if (!aligned4(amax_dev)) return UE5M3_EALIGN;
    return hip_status(ue5m3::launch_amax(x_bf16, numel, amax_dev, clear == 1, stream));
}

ue5m3_status_t ue5m3_quantize_1d_ex(const void* x_bf16, int64_t rows, int64_t cols, int32_t axis,
                                    const float* amax_dev, float target, ue5m3_round_t mode,
                                    uint64_t seed, uint32_t tensor_id, ue5m3_scale_kind_t scale_kind,
                                    int32_t block, uint8_t* payload, uint8_t* scales, float* dec_out,
                                    hipStream_t stream) {
    if (axis != 0 && axis != 1) return UE5M3_EINVAL;
    if (mode != UE5M3_RN && mode != UE5M3_SR) return UE5M3_EINVAL;
    if (scale_kind != UE5M3_SCALE_UE5M3 && scale_kind != UE5M3_SCALE_E4M3 &&
        scale_kind != UE5M3_SCALE_E8M0)
        return UE5M3_EINVAL;
    const bool e8 = scale_kind == UE5M3_SCALE_E8M0;
    if (e8 ? block != 32 : (block != 16 && block != 32)) return UE5M3_EINVAL;
    if (!e8 && (amax_dev == nullptr || !valid_target(target))) return UE5M3_EINVAL;
    if (rows < 0 || cols < 0) return UE5M3_ESHAPE;
    if (axis == 1 && cols % block != 0) return UE5M3_ESHAPE;
    if (axis == 0 && (rows % block != 0 || cols % 2 != 0)) return UE5M3_ESHAPE;
    if ((amax_dev != nullptr && !aligned4(amax_dev)) || (dec_out != nullptr && !aligned4(dec_out)))
        return UE5M3_EALIGN;
    if (rows == 0 || cols == 0) return UE5M3_OK;
    if (x_bf16 == nullptr || payload == nullptr || scales == nullptr) return UE5M3_EINVAL;
    if (!aligned16(x_bf16) || !aligned16(payload) || !aligned16(scales)) return UE5M3_EALIGN;
    const bool sr = mode == UE5M3_SR;
    const ue5m3::ScaleKind fmt = static_cast<ue5m3::ScaleKind>(scale_kind);
    hipError_t e;
    if (axis == 1)
        e = ue5m3::launch_quant_rows(fmt, block, x_bf16, rows, cols, amax_dev, target, sr, seed, tensor_id,
                                     payload, scales, dec_out, stream);
    else
        e = ue5m3::launch_quant_cols(fmt, block, x_bf16, rows, cols, amax_dev, target, sr, seed, tensor_id,
                                     payload, scales, dec_out, stream);
    return hip_status(e);
}

ue5m3_status_t ue5m3_amax_sample_rht(ue5m3_amax_state_t* st, const void* x_bf16, int64_t rows,
                                     int64_t cols, uint32_t sign_mask, int64_t step, int32_t* refreshed,
                                     hipStream_t stream) {
    if (st == nullptr || st->amax_dev == nullptr || st->period < 0 || sign_mask > 0xFFFFu)
        return UE5M3_EINVAL;
    if (rows < 0 || cols < 0 || rows % 16 != 0 || cols % 2 != 0) return UE5M3_ESHAPE;
    const bool empty = rows == 0 || cols == 0;
    if (!empty && x_bf16 == nullptr) return UE5M3_EINVAL;
    if ((!empty && !aligned16(x_bf16)) || !aligned4(st->amax_dev)) return UE5M3_EALIGN;
    const bool refresh = !st->has_cache ||
                         (st->period > 0 && step - st->last_refresh >= (int64_t)st->period);
    if (refreshed != nullptr) *refreshed = refresh ? 1 : 0;
    if (!refresh) return UE5M3_OK;
    const hipError_t e = ue5m3::launch_amax_rht(x_bf16, rows, cols, sign_mask, st->amax_dev, stream);
    if (e != hipSuccess) return UE5M3_EHIP;
    st->has_cache = 1;
    st->last_refresh = step;
    return UE5M3_OK;
}

ue5m3_status_t ue5m3_quantize_cols_rht(const void* x_bf16, int64_t rows, int64_t cols,
                                       const float* amax_dev, float target, ue5m3_round_t mode,
                                       uint64_t seed, uint32_t tensor_id, uint32_t sign_mask,
                                       uint8_t* payload_t, uint8_t* scales_t, float* dec_out,
                                       hipStream_t stream) {
    if (mode != UE5M3_RN && mode != UE5M3_SR) return UE5M3_EINVAL;
    if (amax_dev == nullptr || !valid_target(target) || sign_mask > 0xFFFFu) return UE5M3_EINVAL;
    if (rows < 0 || cols < 0 || rows % 16 != 0 || cols % 2 != 0) return UE5M3_ESHAPE;
    if (!aligned4(amax_dev) || (dec_out != nullptr && !aligned4(dec_out))) return UE5M3_EALIGN;
    if (rows == 0 || cols == 0) return UE5M3_OK;
    if (x_bf16 == nullptr || payload_t == nullptr || scales_t == nullptr) return UE5M3_EINVAL;
    if (!aligned16(x_bf16) || !aligned16(payload_t) || !aligned16(scales_t)) return UE5M3_EALIGN;
    return hip_status(ue5m3::launch_quant_cols_rht(x_bf16, rows, cols, amax_dev, target, mode == UE5M3_SR,
                                                   seed, tensor_id, sign_mask, payload_t, scales_t,
                                                   dec_out, stream));
}

ue5m3_status_t ue5m3_quantize_1d(const void* x_bf16, int64_t rows, int64_t cols, int32_t axis,
                                 const float* amax_dev, float target, ue5m3_round_t mode,
                                 uint64_t seed, uint32_t tensor_id, uint8_t* payload,
                                 uint8_t* scales, float* dec_out, hipStream_t stream) {
    return ue5m3_quantize_1d_ex(x_bf16, rows, cols, axis, amax_dev, target, mode, seed, tensor_id,
                                UE5M3_SCALE_UE5M3, 16, payload, scales, dec_out, stream);
}

ue5m3_status_t ue5m3_quantize_2d_ex(const void* w_bf16, int64_t rows, int64_t cols,
                                    const float* amax_dev, float target, ue5m3_round_t mode,
                                    uint64_t seed, uint32_t tensor_id, ue5m3_scale_kind_t scale_kind,
                                    int32_t block, uint8_t* payload, uint8_t* scales, uint8_t* payload_t,
                                    uint8_t* scales_t, float* dec_out, hipStream_t stream) {
    if (mode != UE5M3_RN && mode != UE5M3_SR) return UE5M3_EINVAL;
    if (scale_kind != UE5M3_SCALE_UE5M3 && scale_kind != UE5M3_SCALE_E4M3) return UE5M3_EINVAL;
    if (block != 16 && block != 32) return UE5M3_EINVAL;
    if (amax_dev == nullptr || !valid_target(target)) return UE5M3_EINVAL;
    if (rows < 0 || cols < 0 || rows % block != 0 || cols % block != 0) return UE5M3_ESHAPE;
    if (!aligned4(amax_dev) || (dec_out != nullptr && !aligned4(dec_out))) return UE5M3_EALIGN;
    if (rows == 0 || cols == 0) return UE5M3_OK;
    if (w_bf16 == nullptr || payload == nullptr || scales == nullptr) return UE5M3_EINVAL;
    if (!aligned16(w_bf16) || !aligned16(payload) || !aligned16(scales) ||
        (payload_t != nullptr && !aligned16(payload_t)) ||
        (scales_t != nullptr && !aligned16(scales_t)))
        return UE5M3_EALIGN;
    return hip_status(ue5m3::launch_quant_tiles(static_cast<ue5m3::ScaleKind>(scale_kind), block, w_bf16, rows,
                                                cols, amax_dev, target, mode == UE5M3_SR, seed,
                                                tensor_id, payload, scales, payload_t, scales_t,
                                                dec_out, stream));
}

ue5m3_status_t ue5m3_quantize_2d(const void* w_bf16, int64_t rows, int64_t cols,
                                 const float* amax_dev, float target, ue5m3_round_t mode,
                                 uint64_t seed, uint32_t tensor_id, uint8_t* payload,
                                 uint8_t* scales, uint8_t* payload_t, uint8_t* scales_t,
                                 float* dec_out, hipStream_t stream) {
    return ue5m3_quantize_2d_ex(w_bf16, rows, cols, amax_dev, target, mode, seed, tensor_id,
                                UE5M3_SCALE_UE5M3, 16, payload, scales, payload_t, scales_t, dec_out,
                                stream);
}

ue5m3_status_t ue5m3_quantize_dual(const void* x_bf16, int64_t rows, int64_t cols,
                                   const float* amax_dev, float target, ue5m3_round_t mode,
                                   uint64_t seed, uint32_t tensor_id_r, uint32_t tensor_id_c,
                                   int32_t scale_kind, uint8_t* payload_r, uint8_t* scales_r,
                                   uint8_t* payload_c, uint8_t* scales_c, float* dec_out,
                                   hipStream_t stream) {
    if (mode != UE5M3_RN && mode != UE5M3_SR) return UE5M3_EINVAL;
    if (scale_kind != UE5M3_SCALE_UE5M3 && scale_kind != UE5M3_SCALE_E4M3) return UE5M3_EINVAL;
    if (amax_dev == nullptr || !valid_target(target)) return UE5M3_EINVAL;
    if (rows < 0 || cols < 0 || rows % 16 != 0 || cols % 16 != 0) return UE5M3_ESHAPE;
    if (!aligned4(amax_dev) || (dec_out != nullptr && !aligned4(dec_out))) return UE5M3_EALIGN;
    if (rows == 0 || cols == 0) return UE5M3_OK;
    if (x_bf16 == nullptr || payload_r == nullptr || scales_r == nullptr || payload_c == nullptr ||
        scales_c == nullptr)
        return UE5M3_EINVAL;
    if (!aligned16(x_bf16) || !aligned16(payload_r) || !aligned16(scales_r) || !aligned16(payload_c) ||
        !aligned16(scales_c))
        return UE5M3_EALIGN;
    return hip_status(ue5m3::launch_quant_dual(static_cast<ue5m3::ScaleKind>(scale_kind), x_bf16, rows, cols,
                                               amax_dev, target, mode == UE5M3_SR, seed, tensor_id_r,
                                               tensor_id_c, payload_r, scales_r, payload_c, scales_c,
                                               dec_out, stream));
}

ue5m3_status_t ue5m3_gemm_ex(ue5m3_layout_t layout, int64_t M, int64_t N, int64_t K,
                             const uint8_t* a, const uint8_t* a_scales, ue5m3_blocking_t a_blk,
                             const float* a_dec, const uint8_t* b, const uint8_t* b_scales,
                             ue5m3_blocking_t b_blk, const float* b_dec, void* c, ue5m3_out_t c_type,
                             ue5m3_scale_kind_t scale_kind, hipStream_t stream) {
    if (layout != UE5M3_NT && layout != UE5M3_NN && layout != UE5M3_TN) return UE5M3_ELAYOUT;
    if (scale_kind != UE5M3_SCALE_UE5M3 && scale_kind != UE5M3_SCALE_E4M3 &&
        scale_kind != UE5M3_SCALE_E8M0)
        return UE5M3_EINVAL;
    const bool e8 = scale_kind == UE5M3_SCALE_E8M0;
    int block = 16;
    ue5m3::BScale bmode = ue5m3::BScale::Row;
    const ue5m3_status_t bst = gemm_blockings(layout, a_blk, b_blk, e8, &block, &bmode);
    if (bst != UE5M3_OK) return bst;
    const bool tiled = bmode != ue5m3::BScale::Row;
    if (c_type != UE5M3_OUT_F32 && c_type != UE5M3_OUT_BF16) return UE5M3_EINVAL;
    if (M < 0 || N < 0 || K < 0 || K % block != 0) return UE5M3_ESHAPE;
    if (tiled && N % block != 0) return UE5M3_ESHAPE;
    if (e8) {
        const int64_t lim = (int64_t)1 << 31;
        if (K % 256 != 0 || M * (K / 2) >= lim || N * (K / 2) >= lim || 4 * M * N >= lim)
            return UE5M3_ESHAPE;
    }
    if (M == 0 || N == 0) return UE5M3_OK;
    if (c == nullptr || a_dec == nullptr || b_dec == nullptr) return UE5M3_EINVAL;
    if (K > 0 && (a == nullptr || a_scales == nullptr || b == nullptr || b_scales == nullptr))
        return UE5M3_EINVAL;
    if (!aligned16(c) || !aligned4(a_dec) || !aligned4(b_dec)) return UE5M3_EALIGN;
    if (K > 0 && (!aligned16(a) || !aligned16(b) || !aligned16(a_scales) || !aligned16(b_scales)))
        return UE5M3_EALIGN;
    const bool bf = c_type == UE5M3_OUT_BF16;
    if (e8) {
        if (K == 0)   // no products: zeros, through the general kernel
            return hip_status(ue5m3::launch_gemm(ue5m3::BScale::Row, 1.0f, M, N, K, a, a_scales, a_dec,
                                                 b, b_scales, b_dec, c, bf, stream));
        return hip_status(ue5m3::launch_gemm_mx(M, N, K, a, a_scales, a_dec, b, b_scales, b_dec, c, bf,
                                                stream));
    }
    // UE5M3 codes decode with the operands scaled by 2^-3 (alpha * 2^6); E4M3
    // codes read as UE5M3 are value / 2^8, so alpha * 2^22.
    const float amul = scale_kind == UE5M3_SCALE_E4M3 ? 4194304.0f : 64.0f;
    if (block == 32)
        return hip_status(ue5m3::launch_gemm_b32(bmode, amul, false, 0.0f, M, N, K, a, a_scales, a_dec, b,
                                                 b_scales, b_dec, c, bf, stream));
    return hip_status(ue5m3::launch_gemm(bmode, amul, M, N, K, a, a_scales, a_dec, b, b_scales, b_dec, c,
                                         bf, stream));
}

ue5m3_status_t ue5m3_gemm_pm(ue5m3_layout_t layout, int64_t M, int64_t N, int64_t K,
                             const uint8_t* a, const uint8_t* a_scales, ue5m3_blocking_t a_blk,
                             const float* a_dec, const uint8_t* b, const uint8_t* b_scales,
                             ue5m3_blocking_t b_blk, const float* b_dec, void* c, ue5m3_out_t c_type,
                             ue5m3_scale_kind_t scale_kind, int32_t grid_d, hipStream_t stream) {
    if (layout != UE5M3_NT && layout != UE5M3_NN && layout != UE5M3_TN) return UE5M3_ELAYOUT;
    if (scale_kind != UE5M3_SCALE_UE5M3 && scale_kind != UE5M3_SCALE_E4M3) return UE5M3_EINVAL;
    int block = 16;
    ue5m3::BScale bmode = ue5m3::BScale::Row;
    const ue5m3_status_t bst = gemm_blockings(layout, a_blk, b_blk, false, &block, &bmode);
    if (bst != UE5M3_OK) return bst;
    const bool tiled = bmode != ue5m3::BScale::Row;
    if (c_type != UE5M3_OUT_F32 && c_type != UE5M3_OUT_BF16) return UE5M3_EINVAL;
    if (grid_d < 0 || grid_d > (1 << 30) || (grid_d & (grid_d - 1)) != 0) return UE5M3_EINVAL;
    if (M < 0 || N < 0 || K < 0 || K % block != 0) return UE5M3_ESHAPE;
    if (tiled && N % block != 0) return UE5M3_ESHAPE;
    if (M == 0 || N == 0) return UE5M3_OK;
    if (c == nullptr || a_dec == nullptr || b_dec == nullptr) return UE5M3_EINVAL;
    if (K > 0 && (a == nullptr || a_scales == nullptr || b == nullptr || b_scales == nullptr))
        return UE5M3_EINVAL;
    if (!aligned16(c) || !aligned4(a_dec) || !aligned4(b_dec)) return UE5M3_EALIGN;
    if (K > 0 && (!aligned16(a) || !aligned16(b) || !aligned16(a_scales) || !aligned16(b_scales)))
        return UE5M3_EALIGN;
    const float amul = scale_kind == UE5M3_SCALE_E4M3 ? 4194304.0f : 64.0f;
    const bool bf = c_type == UE5M3_OUT_BF16;
    if (block == 32)
        return hip_status(ue5m3::launch_gemm_b32(bmode, amul, true, (float)grid_d, M, N, K, a, a_scales, a_dec,
                                                 b, b_scales, b_dec, c, bf, stream));
    return hip_status(ue5m3::launch_gemm_pm(bmode, amul, (float)grid_d, M, N, K, a, a_scales, a_dec, b,
                                            b_scales, b_dec, c, bf, stream));
}

ue5m3_status_t ue5m3_gemm(ue5m3_layout_t layout, int64_t M, int64_t N, int64_t K,
                          const uint8_t* a, const uint8_t* a_scales, ue5m3_blocking_t a_blk,
                          const float* a_dec, const uint8_t* b, const uint8_t* b_scales,
                          ue5m3_blocking_t b_blk, const float* b_dec, void* c, ue5m3_out_t c_type,
                          hipStream_t stream) {
    // blocks of 16 only; the other checks are ue5m3_gemm_ex's
    int len = 0;
    Orient o = Orient::Row;
    if (layout == UE5M3_NT || layout == UE5M3_NN || layout == UE5M3_TN) {
        if (!blocking_of(a_blk, len, o) || len != 16 || !blocking_of(b_blk, len, o) || len != 16)
            return UE5M3_EINVAL;
    }
    return ue5m3_gemm_ex(layout, M, N, K, a, a_scales, a_blk, a_dec, b, b_scales, b_blk, b_dec, c, c_type,
                         UE5M3_SCALE_UE5M3, stream);
}

ue5m3_status_t ue5m3_gemm_noalloc(ue5m3_layout_t layout, int64_t M, int64_t N, int64_t K,
                                  const uint8_t* a, const uint8_t* a_scales, ue5m3_blocking_t a_blk,
                                  const float* a_dec, const uint8_t* b, const uint8_t* b_scales,
                                  ue5m3_blocking_t b_blk, const float* b_dec, void* c, ue5m3_out_t c_type,
                                  hipStream_t stream) {
    // the checks of ue5m3_gemm (blocks of 16, UE5M3)
    if (layout != UE5M3_NT && layout != UE5M3_NN && layout != UE5M3_TN) return UE5M3_ELAYOUT;
    int len = 0;
    Orient o = Orient::Row;
    if (!blocking_of(a_blk, len, o) || len != 16 || !blocking_of(b_blk, len, o) || len != 16)
        return UE5M3_EINVAL;
    int block = 16;
    ue5m3::BScale bmode = ue5m3::BScale::Row;
    const ue5m3_status_t bst = gemm_blockings(layout, a_blk, b_blk, false, &block, &bmode);
    if (bst != UE5M3_OK) return bst;
    if (c_type != UE5M3_OUT_F32 && c_type != UE5M3_OUT_BF16) return UE5M3_EINVAL;
    if (M < 0 || N < 0 || K < 0 || K % 16 != 0) return UE5M3_ESHAPE;
    if (bmode != ue5m3::BScale::Row && N % 16 != 0) return UE5M3_ESHAPE;
    if (M == 0 || N == 0) return UE5M3_OK;
    if (c == nullptr || a_dec == nullptr || b_dec == nullptr) return UE5M3_EINVAL;
    if (K > 0 && (a == nullptr || a_scales == nullptr || b == nullptr || b_scales == nullptr))
        return UE5M3_EINVAL;
    if (!aligned16(c) || !aligned4(a_dec) || !aligned4(b_dec)) return UE5M3_EALIGN;
    if (K > 0 && (!aligned16(a) || !aligned16(b) || !aligned16(a_scales) || !aligned16(b_scales)))
        return UE5M3_EALIGN;
    ue5m3::FixedScratch fx{nullptr, 0};
    if (ue5m3::noalloc_scratch(&fx) != hipSuccess) return UE5M3_EHIP;
    const hipError_t e = ue5m3::launch_gemm(bmode, 64.0f, M, N, K, a, a_scales, a_dec, b, b_scales, b_dec, c,
                                            c_type == UE5M3_OUT_BF16, stream, &fx);
    if (e == hipErrorOutOfMemory) return UE5M3_ESCRATCH;
    return hip_status(e);
}

}  // extern "C"
