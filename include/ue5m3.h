/*
 * ue5m3.h -- C ABI of the UE5M3 FP4 quantize-and-GEMM library for MI355X
 * (gfx950).
 *
 * Implements the per-linear hot path of "UE5M3 FP4 Block Scaling for Stable
 * Language Model Pretraining" (arXiv 2609.02846): E2M1 payloads in blocks of
 * 16 with unsigned E5M3 (UE5M3) block scales -- 1D along the contraction
 * dimension for activations and gradients, 2D 16x16 tiles for weights --
 * under a periodic sample-and-hold tensor amax, stochastic rounding of the
 * upstream gradient only, and the decoded-operand fprop / dgrad / wgrad
 * GEMMs.
 *
 * Conventions shared by every call
 * --------------------------------
 * - All tensor pointers are DEVICE pointers owned by the caller, who
 *   allocates and frees them.  Every pointer must be 16-byte aligned.  The
 *   only memory the library allocates itself is a set of workspaces, one of
 *   each kind per (device, stream): the split-tile partials of ue5m3_gemm,
 *   the expanded block-32 scales of ue5m3_gemm_ex / ue5m3_gemm_pm, and
 *   16 KiB of per-workgroup partial maxima for the amax calls.  A workspace
 *   is allocated (hipMalloc) by the first call on that pair that needs it,
 *   or needs a larger one; a replaced workspace is never freed before the
 *   process ends, so work already enqueued or captured in a graph keeps a
 *   valid buffer.  Calls on one stream use a workspace in stream order;
 *   streams are told apart by handle value, so a stream should be destroyed
 *   only after its work has completed, and at most 64 (device, stream)
 *   pairs can hold workspaces (a further pair gets UE5M3_EHIP).
 *   ue5m3_gemm_noalloc uses no workspace (see there).  Besides these the
 *   library keeps only caches of device properties.  The library
 *   may be called from several host threads at once.
 * - Stream capture: a call made while `stream` is capturing that would have
 *   to allocate or grow a workspace returns UE5M3_EHIP and enqueues
 *   nothing; run the same call once before capturing (no library call
 *   records a memset node).  A captured graph uses the workspaces of the
 *   stream it was captured on: replay it on that stream, or never while a
 *   call on that stream may run.
 * - bf16 tensors are dense row-major [rows, cols] arrays of 16-bit words.
 * - Payloads pack two E2M1 nibbles per byte along a row: byte [r, c/2] holds
 *   element (r, c) in its low nibble and (r, c+1) in its high nibble.
 *   Nibble = sign << 3 | magnitude code, magnitudes {0, .5, 1, 1.5, 2, 3, 4, 6}.
 * - Scale bytes are UE5M3 codes (value (1 + m/8) 2^(e-15) for exponent field
 *   e >= 1, m 2^-17 for e = 0), stored row-major as described per call.
 * - Every call only enqueues work on `stream` (a hipStream_t; 0 is the null
 *   stream) and returns without synchronizing the stream or the device (a
 *   workspace allocation is a hipMalloc, see above).  Argument errors are
 *   detected on the host before anything is enqueued; then nothing is
 *   written.
 * - Inputs must not be NaN (the nibbles and codes of NaN elements are
 *   unspecified); +-Inf is quantized like any magnitude above the E2M1 and
 *   UE5M3 ranges (saturation).
 * - No C++ exception crosses this interface.
 */
#ifndef UE5M3_H
#define UE5M3_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    UE5M3_OK = 0,
    UE5M3_EINVAL = 1,   /* null pointer, bad enum, bad target/period    */
    UE5M3_ESHAPE = 2,   /* negative size or size not a required multiple */
    UE5M3_EALIGN = 3,   /* pointer not 16-byte aligned                   */
    UE5M3_ELAYOUT = 4,  /* unknown GEMM layout, or an operand blocking
                           that does not run along the contraction      */
    UE5M3_EHIP = 5,     /* a HIP launch or runtime call failed           */
    UE5M3_ESCRATCH = 6  /* more scratch than ue5m3_gemm_noalloc holds    */
} ue5m3_status_t;

typedef enum { UE5M3_RN = 0, UE5M3_SR = 1 } ue5m3_round_t;

typedef enum { UE5M3_NT = 0, UE5M3_NN = 1, UE5M3_TN = 2 } ue5m3_layout_t;

typedef enum { UE5M3_OUT_F32 = 0, UE5M3_OUT_BF16 = 1 } ue5m3_out_t;

/*
 * Blocking of a quantized GEMM operand: along which dimension of its source
 * tensor s [R, C] the scale blocks run, and hence how the quantizer stored
 * it (eq:microscaling: a block scale is shared by consecutive elements of
 * one contraction; Sec. 4.3 and Table 5: each GEMM needs its operands
 * blocked along its own contraction dimension).
 *   UE5M3_ROW16   blocks of 16 along a row (ue5m3_quantize_1d, axis 1):
 *                 payload [R, C/2], scales [R, C/16].
 *   UE5M3_COL16T  blocks of 16 down a column (ue5m3_quantize_1d, axis 0),
 *                 stored transposed: payload [C, R/2], scales [C, R/16].
 *   UE5M3_TILE16  16 x 16 tiles (ue5m3_quantize_2d): for a contraction along
 *                 the rows of s the payload [R, C/2] and scales [R/16, C/16];
 *                 for a contraction down its columns the transposed copy
 *                 payload_t [C, R/2] and scales_t [C/16, R/16].
 *   UE5M3_ROW32, UE5M3_COL32T, UE5M3_TILE32: the same with blocks of 32
 *                 (32 x 32 tiles), for ue5m3_gemm_ex and ue5m3_gemm_pm.
 * In every case the operand as passed is contraction-contiguous: a row of
 * the payload holds consecutive contraction indices.
 */
typedef enum {
    UE5M3_ROW16 = 0,
    UE5M3_COL16T = 1,
    UE5M3_TILE16 = 2,
    UE5M3_ROW32 = 3,
    UE5M3_COL32T = 4,
    UE5M3_TILE32 = 5
} ue5m3_blocking_t;

/*
 * Sample-and-hold state of one operand's tensor reference (paper Sec. 4.1,
 * eq:delayed-amax).  Plain host data plus one caller-owned device float.
 *   amax_dev      device float receiving the sampled amax (fp32 bits of
 *                 max |x|); read by the quantizers.
 *   last_refresh  optimizer step of the last refresh (tau).
 *   period        refresh period D in optimizer steps (50 in the paper's
 *                 recipe; 1 = current scaling; 0 = measure once, then hold
 *                 until reset: the inference policy for loaded weights, Sec.
 *                 "Inference with delayed scaling").
 *   has_cache     0 until the first refresh; reset to 0 on resume (the
 *                 paper's caches are not checkpointed).
 */
typedef struct {
    float*  amax_dev;
    int64_t last_refresh;
    int32_t period;
    int32_t has_cache;
} ue5m3_amax_state_t;

/* Initialise `st` with an empty cache.  EINVAL if st or amax_dev is null or
 * period < 0; EALIGN if amax_dev is not 4-byte aligned. */
ue5m3_status_t ue5m3_amax_state_init(ue5m3_amax_state_t* st, float* amax_dev,
                                     int32_t period);

/* Empty the cache so that the next ue5m3_amax_sample refreshes (simulated
 * process restart / resume).  A null st is ignored. */
void ue5m3_amax_state_reset(ue5m3_amax_state_t* st);

/* Hold the reference now in *st->amax_dev for good: has_cache = 1 and
 * period = 0, so ue5m3_amax_sample refreshes again only after a reset (the
 * calibrated-frozen inference policy, Table tab:inference-scale-summary).
 * The caller has filled *amax_dev first, e.g. with ue5m3_amax_accumulate
 * over calibration batches.  A null st is ignored. */
void ue5m3_amax_state_freeze(ue5m3_amax_state_t* st);

/*
 * Running tensor amax for calibration (App. "Inference-Scale Sensitivity":
 * the largest activation amax over calibration data).  Enqueues
 * *amax_dev = max(clear ? 0 : *amax_dev, max_i |x_i|) for the bf16 tensor x
 * (numel elements).  With clear = 0, *amax_dev must already hold a
 * non-negative finite float (from an earlier call with clear = 1).
 * EINVAL: null amax_dev, null x with numel > 0, clear not 0 or 1;
 * ESHAPE: numel < 0; EALIGN: x not 16-byte or amax_dev not 4-byte aligned.
 */
ue5m3_status_t ue5m3_amax_accumulate(const void* x_bf16, int64_t numel, float* amax_dev,
                                     int32_t clear, hipStream_t stream);

/*
 * Randomized Hadamard transform of the weight-gradient operands (the "UE5M3
 * with Transformer Engine settings" recipe: paper Table 6, Sec. 2).  The
 * transform replaces every block of 16 consecutive rows (tokens) of each
 * column of a bf16 matrix x [rows, cols] by y = (1/4) H16 diag(s) x_block,
 * H16[i][j] = (-1)^popcount(i & j), s_i = -1 where bit i of sign_mask is set,
 * evaluated in binary32 as sign flips, butterfly stages h = 1, 2, 4, 8
 * ((u_i, u_{i+h}) <- (u_i + u_{i+h}, u_i - u_{i+h}) for i with bit h clear,
 * one rounding each) and an exact 1/4 scaling.  The same sign_mask must be
 * used for both operands of one weight-gradient product (X and dY), which
 * leaves dY^T X unchanged in exact arithmetic.  The paper fixes neither the
 * size nor the signs; the caller draws the mask.
 *
 * ue5m3_amax_sample_rht: ue5m3_amax_sample for the transformed tensor (its
 * amax is the reference of the transformed operand).  Requires rows % 16 ==
 * 0 and cols % 2 == 0 (ESHAPE), sign_mask < 2^16 (EINVAL).
 */
ue5m3_status_t ue5m3_amax_sample_rht(ue5m3_amax_state_t* st, const void* x_bf16, int64_t rows,
                                     int64_t cols, uint32_t sign_mask, int64_t step, int32_t* refreshed,
                                     hipStream_t stream);

/*
 * COL16 quantization (UE5M3, as ue5m3_quantize_1d with axis 0: payload_t
 * [cols][rows/2], scales_t [cols][rows/16]) of the transformed tensor
 * described at ue5m3_amax_sample_rht, with the held reference *amax_dev of
 * the transformed tensor.  SR words follow each element's position (r, c)
 * in x.  Same status codes as ue5m3_quantize_1d, plus EINVAL for
 * sign_mask >= 2^16.
 */
ue5m3_status_t ue5m3_quantize_cols_rht(const void* x_bf16, int64_t rows, int64_t cols,
                                       const float* amax_dev, float target, ue5m3_round_t mode,
                                       uint64_t seed, uint32_t tensor_id, uint32_t sign_mask,
                                       uint8_t* payload_t, uint8_t* scales_t, float* dec_out,
                                       hipStream_t stream);

/*
 * eq:delayed-amax.  At optimizer step `step`, if the cache is empty or
 * period > 0 and step - last_refresh >= period, enqueue the tensor amax
 * a = max_i |x_i| of the bf16 tensor x (numel elements) into *st->amax_dev,
 * set last_refresh = step, has_cache = 1 and *refreshed = 1; otherwise
 * enqueue nothing and set *refreshed = 0.  The decision uses host integers only (no device read).
 * numel = 0 stores amax 0 (the quantizers then use reference 1).
 * `refreshed` may be null.
 */
ue5m3_status_t ue5m3_amax_sample(ue5m3_amax_state_t* st, const void* x_bf16,
                                 int64_t numel, int64_t step, int32_t* refreshed,
                                 hipStream_t stream);

/*
 * 1D block-16 quantization of a bf16 matrix x [rows, cols] (eq:microscaling,
 * eq:scale-target, Table 5).  With g = *amax_dev (the held reference), T =
 * target and F = 6, each block B computes in binary32 (one round-to-nearest-
 * even per operation): S = T/g, G = 6T/g, u = max|x_B| * S, s = UE5M3(u)
 * (nearest, ties to even, saturating above 61440; a zero code is replaced by
 * the code of 1.0), r = G/s, y_i = x_i * r, and the E2M1 nibble of y_i by
 * round-to-nearest-even (mode RN) or stochastic rounding (mode SR, eq:sr).
 * A reference g that is not positive and finite, or with 6T/g >= 2^110, is
 * replaced by 1.
 *
 * SR draws for source element (r, c) the word (r*cols + c) & 3 of
 * Philox4x32-10 with key (seed lo, seed hi) and counter
 * ((r*cols + c) >> 2 as 64 bits, tensor_id, 0), and rounds the magnitude up
 * iff word < ceil(frac * 2^32), frac = (|y| - q_lo) / (q_hi - q_lo).
 *
 * axis = 1 (blocks along rows; fprop X, dgrad dY):
 *     requires cols % 16 == 0;  payload [rows, cols/2];  scales [rows, cols/16].
 * axis = 0 (blocks down columns; wgrad dY and X re-blocked along tokens):
 *     requires rows % 16 == 0 and cols % 2 == 0.  The output is stored
 *     TRANSPOSED, i.e. as the axis-1 quantization of x^T: payload
 *     [cols, rows/2], scales [cols, rows/16].
 * dec_out (nullable): receives the decode multiplier dec = g / (6T) used by
 *     the GEMM epilogue.
 * target must be finite and > 0 (448 default; 2048 for the wgrad-dY
 * override of Sec. 4.2).
 */
ue5m3_status_t ue5m3_quantize_1d(const void* x_bf16, int64_t rows, int64_t cols,
                                 int32_t axis, const float* amax_dev, float target,
                                 ue5m3_round_t mode, uint64_t seed, uint32_t tensor_id,
                                 uint8_t* payload, uint8_t* scales, float* dec_out,
                                 hipStream_t stream);

/*
 * 2D 16x16 tile quantization of a bf16 weight w [rows, cols] (Sec. 2.3 and
 * Table 5: one scale per 16x16 tile so that the row-wise and column-wise GEMM
 * views share the quantized values).  Same per-block arithmetic as
 * ue5m3_quantize_1d with the block maximum taken over the tile.
 * Requires rows % 16 == 0 and cols % 16 == 0.
 *   payload   [rows, cols/2]
 *   scales    [rows/16, cols/16]
 *   payload_t (nullable) [cols, rows/2]: the same nibbles transposed, the
 *             operand of the dgrad GEMM.
 *   scales_t  (nullable) [cols/16, rows/16]: the tile scales transposed, the
 *             scales of that operand.
 *   dec_out   (nullable) decode multiplier, as above.
 */
ue5m3_status_t ue5m3_quantize_2d(const void* w_bf16, int64_t rows, int64_t cols,
                                 const float* amax_dev, float target,
                                 ue5m3_round_t mode, uint64_t seed, uint32_t tensor_id,
                                 uint8_t* payload, uint8_t* scales, uint8_t* payload_t,
                                 uint8_t* scales_t, float* dec_out, hipStream_t stream);

/*
 * Decoded-operand FP4 GEMM (Sec. 5.1; the three products of Sec. 4.3):
 *     C[m, n] = alpha * sum_k A_hat[m, k] * B_hat[n, k],
 *     alpha = RN(*a_dec * *b_dec),
 * where X_hat = E2M1 value * UE5M3 block scale (held exactly, as fp16 values
 * times 2^-3, on the matrix cores), products are exact and the sum is
 * accumulated in fp32; the order of the fp32 additions is unspecified.  C is
 * a dense row-major [M, N] fp32 array (UE5M3_OUT_F32) or bf16 array
 * (UE5M3_OUT_BF16, round to nearest even of the fp32 result).
 *
 * Workspace: when the 256 x 256 output tiles leave a last, mostly idle wave
 * of workgroups, those tiles are split along K and their fp32 partials are
 * summed (in a fixed order) by a second kernel on the same stream.  The
 * partials live in the library's split workspace for (device, stream) (see
 * the conventions above: allocated or grown on need, never freed while the
 * process runs); such a call returns UE5M3_EHIP if the allocation fails.
 *
 * Each operand is (payload, scales, blocking, dec) and is passed in
 * contraction-contiguous form, as produced by the quantizers for each
 * product of a linear Y = X W^T (X [T,K], W [N,K]); the layout names which
 * dimension of each operand's source is contracted:
 *
 * UE5M3_NT  fprop  Y = X W^T:  M = T, N = N, K = K.  Both sources [rows, K]
 *           are contracted along their rows.
 *     a = quantize_1d(X, axis 1), a_blk = ROW16: payload [M, K/2], scales [M, K/16]
 *     b = quantize_2d(W), b_blk = TILE16:      payload [N, K/2], scales [N/16, K/16]
 *         (or b = quantize_1d(W, axis 1), b_blk = ROW16: scales [N, K/16])
 * UE5M3_NN  dgrad  dX = dY W:   M = T, N = K_w, K = N_w.  A (dY [M, K]) is
 *           contracted along its rows, B (W [K, N]) down its columns.
 *     a = quantize_1d(dY, axis 1), a_blk = ROW16: payload [M, K/2], scales [M, K/16]
 *     b = quantize_2d(W), b_blk = TILE16: payload_t [N, K/2], scales_t [N/16, K/16]
 *         (or b = quantize_1d(W, axis 0), b_blk = COL16T: scales [N, K/16])
 * UE5M3_TN  wgrad  dW = dY^T X: M = N_w, N = K_w, K = T.  Both sources
 *           [K, cols] are contracted down their columns.
 *     a = quantize_1d(dY, axis 0), a_blk = COL16T: payload [M, K/2], scales [M, K/16]
 *     b = quantize_1d(X, axis 0),  b_blk = COL16T: payload [N, K/2], scales [N, K/16]
 *         (or the transposed copy of a 2D quantization of X, b_blk = TILE16)
 *
 * Blocking rule (eq:microscaling, Sec. 4.3): an operand contracted along its
 * source's rows takes ROW16 or TILE16, one contracted down its source's
 * columns takes COL16T or TILE16; A is 1D (ROW16 / COL16T) only.  Any other
 * combination -- e.g. an axis-1 dY passed to TN, or an axis-0 X passed to NT
 * -- returns UE5M3_ELAYOUT before anything is enqueued.  A blocking value
 * outside ue5m3_blocking_t, or one with blocks of 32 here, is UE5M3_EINVAL.
 *
 * Requires M, N, K >= 0, K % 16 == 0, and N % 16 == 0 when b_blk = TILE16.
 * M = 0 or N = 0 writes nothing; K = 0 writes zeros.
 */
ue5m3_status_t ue5m3_gemm(ue5m3_layout_t layout, int64_t M, int64_t N, int64_t K,
                          const uint8_t* a, const uint8_t* a_scales, ue5m3_blocking_t a_blk,
                          const float* a_dec, const uint8_t* b, const uint8_t* b_scales,
                          ue5m3_blocking_t b_blk, const float* b_dec, void* c,
                          ue5m3_out_t c_type, hipStream_t stream);

/*
 * ue5m3_gemm for callers that cannot allocate device memory: code under
 * stream capture, tight serving loops, harnesses that forbid hipMalloc.
 * Same arguments, checks, kernels, split plan and results (bit for bit) as
 * ue5m3_gemm; it calls no hipMalloc, hipFree or other allocating routine.
 * The split-tile partials go to a scratch array of 64 MiB that the library
 * holds once per device from the first call on that device until the process
 * ends (its device address is looked up on that first call).  A call whose
 * split plan needs more than the array -- never on a device of at most 256
 * compute units, where the leftover tiles times their parts never exceed
 * 256 partial tiles of 256 KiB -- returns UE5M3_ESCRATCH and enqueues
 * nothing.  The caller passes every input and output.  All calls on one
 * device share the array and leave their partials in it (nothing in it needs
 * to start at zero): calls that overlap on one device, on two streams or from
 * two threads, race and give undefined results.
 */
ue5m3_status_t ue5m3_gemm_noalloc(ue5m3_layout_t layout, int64_t M, int64_t N, int64_t K,
                                  const uint8_t* a, const uint8_t* a_scales, ue5m3_blocking_t a_blk,
                                  const float* a_dec, const uint8_t* b, const uint8_t* b_scales,
                                  ue5m3_blocking_t b_blk, const float* b_dec, void* c,
                                  ue5m3_out_t c_type, hipStream_t stream);

/*
 * Both 1D blockings of one bf16 tensor x [rows, cols] from a single read:
 * the axis-1 result (payload_r [rows, cols/2], scales_r [rows, cols/16]) and
 * the axis-0 result stored transposed (payload_c [cols, rows/2], scales_c
 * [cols, rows/16]), each identical to what ue5m3_quantize_1d_ex writes for
 * that axis -- with SR words keyed on tensor_id_r for the row blocking and
 * tensor_id_c for the column blocking.  These are the two backward operands
 * of dY (dgrad and wgrad) or the fprop and wgrad operands of X.
 * scale_kind UE5M3 or E4M3 (blocks of 16; EINVAL otherwise).  Requires
 * rows % 16 == 0 and cols % 16 == 0.  dec_out (nullable) as in
 * ue5m3_quantize_1d.
 */
ue5m3_status_t ue5m3_quantize_dual(const void* x_bf16, int64_t rows, int64_t cols,
                                   const float* amax_dev, float target, ue5m3_round_t mode,
                                   uint64_t seed, uint32_t tensor_id_r, uint32_t tensor_id_c,
                                   int32_t scale_kind, uint8_t* payload_r, uint8_t* scales_r,
                                   uint8_t* payload_c, uint8_t* scales_c, float* dec_out,
                                   hipStream_t stream);

/*
 * Comparison block-scale formats (Sec. 2, Table tab:formats: the MXFP4 and
 * NVFP4 arrangements of the same E2M1 payload).
 *   UE5M3_SCALE_UE5M3  the recipe: blocks of 16, UE5M3 scales, tensor scale
 *                      (the calls above).
 *   UE5M3_SCALE_E4M3   blocks of 16 with an E4M3 block scale (OCP E4M3FN:
 *                      bias 7, largest 448 = 0x7E, smallest subnormal 2^-9)
 *                      under the same FP32 tensor scale: the per-block
 *                      arithmetic of ue5m3_quantize_1d with s = E4M3(u)
 *                      (nearest, ties to even, saturating above 448) and
 *                      the zero code replaced by 0x38 (1.0).
 *   UE5M3_SCALE_E8M0   blocks of 32 with a power-of-two E8M0 scale (value
 *                      2^(code - 127)) and no tensor scale: for a block
 *                      maximum a > 0, E = clamp(floor(log2 a) - 2, -127, 127)
 *                      (the OCP microscaling rule; 2 is the exponent of the
 *                      largest E2M1 value), code = E + 127, y_i = x_i * 2^-E
 *                      (exact); a = 0 gives code 0.  amax_dev and target
 *                      are ignored (amax_dev may be null) and dec_out
 *                      receives 1.
 */
typedef enum {
    UE5M3_SCALE_UE5M3 = 0,
    UE5M3_SCALE_E4M3 = 1,
    UE5M3_SCALE_E8M0 = 2
} ue5m3_scale_kind_t;

/*
 * ue5m3_quantize_1d with a scale format.  Blocks are `block` elements long:
 * 16 or 32 for UE5M3 and E4M3 (32 is the block-size control of Sec.
 * "Recipe comparison" and Table tab:results: the same per-block arithmetic
 * over 32 elements, one scale code per 32), 32 for E8M0; EINVAL otherwise.  Layouts as in
 * ue5m3_quantize_1d with 16 replaced by `block` (axis 1: cols % block == 0,
 * scales [rows, cols/block]; axis 0: rows % block == 0, cols % 2 == 0,
 * transposed payload [cols, rows/2] and scales [cols, rows/block]).
 */
ue5m3_status_t ue5m3_quantize_1d_ex(const void* x_bf16, int64_t rows, int64_t cols,
                                    int32_t axis, const float* amax_dev, float target,
                                    ue5m3_round_t mode, uint64_t seed, uint32_t tensor_id,
                                    ue5m3_scale_kind_t scale_kind, int32_t block,
                                    uint8_t* payload, uint8_t* scales, float* dec_out,
                                    hipStream_t stream);

/*
 * ue5m3_quantize_2d with a scale format and tile size: UE5M3 or E4M3 with
 * square tiles of `tile` = 16 or 32 (32: the block-size control; one scale
 * code per 32 x 32 tile).  Layouts as in ue5m3_quantize_2d with 16
 * replaced by `tile` (rows % tile == 0, cols % tile == 0; scales and
 * scales_t [rows/tile, cols/tile] and [cols/tile, rows/tile]).  E8M0
 * weights are quantized in 1D blocks of 32 along each GEMM's contraction
 * dimension instead (ue5m3_quantize_1d_ex on W, axis 1 for fprop and axis 0
 * for dgrad), so E8M0 here is EINVAL, as is any other tile size.
 */
ue5m3_status_t ue5m3_quantize_2d_ex(const void* w_bf16, int64_t rows, int64_t cols,
                                    const float* amax_dev, float target,
                                    ue5m3_round_t mode, uint64_t seed, uint32_t tensor_id,
                                    ue5m3_scale_kind_t scale_kind, int32_t tile,
                                    uint8_t* payload, uint8_t* scales, uint8_t* payload_t,
                                    uint8_t* scales_t, float* dec_out, hipStream_t stream);

/*
 * ue5m3_gemm with a scale format; the block length (16 or 32) is that of
 * the two blockings, which must agree (EINVAL otherwise).  The blocking rule
 * and UE5M3_ELAYOUT are as for ue5m3_gemm, with ROW32 / COL32T / TILE32 in
 * place of ROW16 / COL16T / TILE16.
 *   UE5M3, E4M3, blocks of 16: operands and requirements exactly as for
 *         ue5m3_gemm.
 *   UE5M3, E4M3, blocks of 32 (the block-size control): as for blocks of 16
 *         with 16 replaced by 32 -- A scales [M, K/32], B scales [N, K/32]
 *         (ROW32 / COL32T) or [N/32, K/32] (TILE32) -- and K % 32 == 0,
 *         N % 32 == 0 for TILE32.  The block scales are expanded to one
 *         code per 16 elements (per 16 x 16 tile) in the library's
 *         block-32 workspace for (device, stream) and the block-16 kernels
 *         run, so the results obey the ue5m3_gemm bound.
 *   E8M0 (blocks of 32 only, 1D only: TILE32 is EINVAL): every layout takes
 *         A as [M, K/2] payload with [M, K/32] scales and B as [N, K/2]
 *         payload with [N, K/32] scales, both blocked along the contraction:
 *           NT fprop: a = quantize_1d_ex(X, axis 1) ROW32, b = quantize_1d_ex(W, axis 1) ROW32
 *           NN dgrad: a = quantize_1d_ex(dY, axis 1) ROW32, b = quantize_1d_ex(W, axis 0) COL32T
 *           TN wgrad: a = quantize_1d_ex(dY, axis 0) COL32T, b = quantize_1d_ex(X, axis 0) COL32T
 *         The products run on the gfx950 scaled FP4 matrix instructions,
 *         which apply the E8M0 powers of two themselves.  Requires
 *         K % 256 == 0, and M*K/2, N*K/2 and 4*M*N each below 2^31 (ESHAPE
 *         otherwise); a_dec and b_dec hold the decode multipliers (1 from the
 *         E8M0 quantizers).  Workspace as for ue5m3_gemm.
 */
ue5m3_status_t ue5m3_gemm_ex(ue5m3_layout_t layout, int64_t M, int64_t N, int64_t K,
                             const uint8_t* a, const uint8_t* a_scales, ue5m3_blocking_t a_blk,
                             const float* a_dec, const uint8_t* b, const uint8_t* b_scales,
                             ue5m3_blocking_t b_blk, const float* b_dec, void* c,
                             ue5m3_out_t c_type, ue5m3_scale_kind_t scale_kind,
                             hipStream_t stream);

/*
 * Probe-matched GEMM: the paper's output model of the native FP4 GEMM (Sec.
 * "The observed reduction and product lattice", eq:issue-partial,
 * eq:issue-rz, eq:final-grid; Sec. "Final-grid granularity",
 * eq:grid-denominator) on the same operands as ue5m3_gemm / ue5m3_gemm_ex.
 * For every output, with the decoded operands a_k b_k (E2M1 value times
 * block scale value) in ascending k:
 *   p_j = binary32 round-to-nearest-even of the exact sum of products
 *         k = 64 j .. 64 j + 63,
 *   c_0 = 0, c_{j+1} = binary32 round-toward-zero of c_j + p_j,
 *   y   = alpha * Q_d(c_J), Q_d(c) = RNE(d c) / d (ties to the even
 *         integer), Q_0(c) = c, alpha = dec_a * dec_b in binary32, one
 *         binary32 rounding, then RNE to bf16 for UE5M3_OUT_BF16.
 * Results are exact to this definition for every input (no accumulation
 * tolerance).  grid_d: 0 (no snap) or a power of two up to 2^30 (the paper
 * uses 1024), else EINVAL.  scale_kind: UE5M3 or E4M3 (E8M0: EINVAL);
 * blocks of 16 or 32 as given by the blockings (a scale code's value is the
 * same in every 16-element group it covers, so the 64-product groups and the
 * result are defined as for blocks of 16).  Layouts, blockings, operand
 * shapes, alignment, the block-32 workspace and the other status codes as
 * ue5m3_gemm_ex.  The K
 * loop runs in one workgroup per output tile in ascending k (the
 * toward-zero chain is order dependent), so this call is several times
 * slower than ue5m3_gemm.
 */
ue5m3_status_t ue5m3_gemm_pm(ue5m3_layout_t layout, int64_t M, int64_t N, int64_t K,
                             const uint8_t* a, const uint8_t* a_scales, ue5m3_blocking_t a_blk,
                             const float* a_dec, const uint8_t* b, const uint8_t* b_scales,
                             ue5m3_blocking_t b_blk, const float* b_dec, void* c,
                             ue5m3_out_t c_type, ue5m3_scale_kind_t scale_kind,
                             int32_t grid_d, hipStream_t stream);

/* Static description of a status code. */
const char* ue5m3_status_string(ue5m3_status_t status);

/* Library ABI version (major * 10000 + minor * 100 + patch). */
int32_t ue5m3_version(void);

#ifdef __cplusplus
}
#endif

#endif /* UE5M3_H */
