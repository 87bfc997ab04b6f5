/*
 * libwinof4 -- integer Winograd F(4x4, 3x3) convolution with tap-wise
 * power-of-two quantization on AMD Instinct MI355X (gfx950).
 *
 * Method: arxiv 2209.12982, Sec. III.  For one output channel and one 4x4
 * output tile,
 *     Y = A^T ( S_BG (.) sum_ci q(B^T d B (/) S_B) (.) q(G f G^T (/) S_G) ) A
 * with per-tap (6x6) power-of-two scales S_B = 2^e_B, S_G = 2^e_G, S_BG =
 * S_B (.) S_G, and q the int8 quantizer of Eq. quant.  The transform matrices
 * are the F(4x4,3x3) ones printed in Sec. II.  Products are accumulated over
 * input channels in int32; the tap scale is applied once, before the back
 * transform (Sec. III, rearranged scheme).
 *
 * Conventions shared by every entry point
 *   - 3x3 kernel, stride 1, zero padding 1, dilation 1, one group: the only
 *     layers the paper sends to Winograd (Sec. III, last paragraph).  Other
 *     geometries are not expressible in this API.
 *   - Tap t = 6*a + b addresses row a, column b of the 6x6 Winograd tile.
 *   - Rounding R(v) = floor(v + 1/2) (round half up) for every rounding; the
 *     int8 quantizer is clamp(R(v / 2^e), -128, 127).  The paper does not
 *     state a tie-break; this is the reading the library implements.
 *   - Input tiles are 6x6 windows at stride 4 over the input padded by one
 *     zero pixel; ceil(H/4) x ceil(W/4) tiles are computed and output pixels
 *     beyond H or W are discarded (zero padding to a multiple of 4, Sec. V).
 *   - Activations are int8, NCHW [N][C][H][W] or NHWC [N][H][W][C], dense.
 *   - "device" pointers are HIP device memory of the current device; "host"
 *     pointers are ordinary CPU memory, read or written during the call only.
 *   - Calls on a stream are asynchronous unless stated; nothing is retained
 *     from a host argument after the call returns.
 *   - Every function validates all arguments before launching anything and
 *     reports failure through its return value; nothing aborts or throws.
 */
#ifndef WINOF4_H
#define WINOF4_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum wino_status {
    WINO_OK = 0,
    WINO_EINVAL = -1,        /* null pointer, negative size, value out of range   */
    WINO_EUNSUPPORTED = -2,  /* a size beyond the library's limits                */
    WINO_ERANGE = -3,        /* plan tables that no integer epilogue can hold     */
    WINO_ENOMEM = -4,        /* device or host allocation failed                  */
    WINO_EWORKSPACE = -5,    /* workspace pointer null or smaller than required   */
    WINO_EHIP = -6           /* a HIP runtime call or kernel launch failed        */
} wino_status;

typedef enum wino_layout { WINO_NCHW = 0, WINO_NHWC = 1 } wino_layout;

/* SPLIT: input transform to a tap-major int8 workspace, then the tap GEMM
 * with the output transform fused into its epilogue (two launches).
 * FUSED: one launch; the input transform runs in the GEMM prologue and no
 * workspace is used.                                                        */
typedef enum wino_variant { WINO_SPLIT = 0, WINO_FUSED = 1 } wino_variant;

typedef struct wino_f4_plan_s* wino_f4_plan_t;   /* opaque, immutable after creation */

/* Which kernel runs the tap GEMM of the SPLIT variant (all give the same,
 * exact result).  RESIDENT keeps all 36 tap accumulators of its block in
 * registers and applies the output transform once at the end, with blocks of
 * 64 channels x 32 tiles (RESIDENT, RESIDENT_64X32), 32 x 32 or 16 x 16 (the
 * _NxM values force a shape).  ROWS streams the taps one row of the 6x6 tile
 * at a time and folds each row into the output as it completes, which allows
 * 64 x 64 blocks.  WAVES (F4, 8-bit, 32-bit epilogue; forced only) splits a
 * 64 x 64 block between four 32x32x32-MFMA waves and eight waves that copy
 * operands and keep the output rows, persistent over the blocks.  AUTO picks
 * ROWS when its blocks fill the device and the 32-bit epilogue applies, else
 * RESIDENT_64X32.  ROWS_STREAMK (forced only: measured slower than ROWS)
 * is ROWS with the blocks of its last, partial round of workgroups split by
 * stages over every compute unit (stream-K): each workgroup runs an equal
 * share of those blocks' stages, leaves partial sums in the workspace and the
 * last to finish a block adds them up.  It needs the larger workspace that
 * wino_f4_workspace_bytes then reports, and runs unsplit in a smaller one. */
typedef enum wino_tap_kernel {
    WINO_TAP_AUTO = 0,
    WINO_TAP_RESIDENT = 1,
    WINO_TAP_ROWS = 2,
    WINO_TAP_RESIDENT_64X32 = 3,
    WINO_TAP_RESIDENT_32X32 = 4,
    WINO_TAP_RESIDENT_16X16 = 5,
    WINO_TAP_WAVES = 6,
    WINO_TAP_ROWS_STREAMK = 7
} wino_tap_kernel;

/*
 * wino_f4_plan -- the offline step: weight transform U = G f G^T (Eq.
 * winograd), tap-wise power-of-two weight quantization (Sec. III-B,
 * straight-forward power-of-two rule), and the per-tap alignment of
 * S_BG (Sec. III, rearranged scheme), uploaded for stationary reuse by every
 * later convolution (the "weights transformed once, kept stationary" dataflow
 * of Sec. IV-B2).
 *
 *   out        receives the new plan (host pointer to a handle).
 *   w_oihw     host fp32 [cout][cin][3][3].  U is computed exactly (no
 *              floating-point rounding), then Uq = clamp(R(U / 2^e_G)).
 *   cin, cout  channel counts, 1 .. 65536 each.
 *   in_exp     host int8 [36]: e_B[t] in [0, 15], the input tap exponents
 *              (S_B = 2^e_B); see wino_f4_calibrate_input.
 *   w_exp      host int8 [36] explicit e_G[t] in [-126, 126], or NULL for
 *              max-abs calibration: e_G[t] = smallest e with
 *              max_{co,ci} |U_t| <= 128 * 2^e (0 for an all-zero tap).
 *   bias       host int32 [cout] in units of 2^e_o (see below), or NULL for 0.
 *   out_shift  output requantization shift in [0, 62]:
 *              out = clamp(R((Y + bias) / 2^out_shift), -128, 127).
 *   relu       0 or 1: if 1, out = max(out, 0).
 *   stream     stream for the upload; the call returns after the upload has
 *              completed, so the plan is usable on any stream afterwards.
 *
 * Exponent bookkeeping: e[t] = e_B[t] + e_G[t], e_o = min_t e[t], and
 * sh[t] = e[t] - e_o.  The tap GEMM result of tap t is multiplied by 2^sh[t]
 * exactly, so Y is an exact integer and the real-valued output is Y * 2^e_o.
 * The plan bounds every intermediate of the output transform; it selects a
 * 32-bit epilogue when the bound is below 2^31, a 64-bit one when below 2^62,
 * and returns WINO_ERANGE otherwise.
 * Errors: WINO_EINVAL (null out/w_oihw/in_exp, values out of range),
 * WINO_ERANGE, WINO_ENOMEM, WINO_EHIP.  On error *out is set to NULL.
 */
wino_status wino_f4_plan(wino_f4_plan_t* out, const float* w_oihw, int32_t cin, int32_t cout,
                         const int8_t* in_exp, const int8_t* w_exp, const int32_t* bias,
                         int32_t out_shift, int32_t relu, hipStream_t stream);

/*
 * wino_f4_plan_tables -- the host arithmetic of wino_f4_plan alone, with no
 * device work: for the same arguments it writes e_g[36], sh[36], e_o,
 * epilogue_bits and uq [36][cin][cout] (host pointers, any may be NULL).
 * Lets a plan be inspected on a machine without a GPU.  Errors as for
 * wino_f4_plan except WINO_EHIP.
 */
wino_status wino_f4_plan_tables(const float* w_oihw, int32_t cin, int32_t cout, const int8_t* in_exp,
                                const int8_t* w_exp, const int32_t* bias, int32_t out_shift, int8_t* e_g,
                                int8_t* sh, int32_t* e_o, int32_t* epilogue_bits, int8_t* uq);

/*
 * wino_f4_plan_set_tap_kernel -- choose the tap-GEMM kernel (wino_tap_kernel)
 * for later SPLIT convolutions with this plan.  ROWS applies to output
 * convolutions with the 32-bit epilogue (else the RESIDENT choice is made);
 * calibration and debug exports always use the 64 x 32 RESIDENT shape.  Not
 * to be called while a convolution with the plan is being enqueued on
 * another thread.
 * Errors: WINO_EINVAL (null plan, unknown kind).
 */
wino_status wino_f4_plan_set_tap_kernel(wino_f4_plan_t plan, int32_t kind);

/*
 * wino_select_algorithm -- per-layer choice between the two Winograd
 * transforms and direct convolution (the paper's point that the best
 * algorithm depends on the layer, Sec. V: F2 for small spatial sizes, F4 for
 * large ones).  Host only, no device work; a fixed rule from measurements on
 * MI355X: DIRECT for NHWC layers below 2^27 direct-equivalent operations
 * (there the two Winograd launches cost more than the whole direct
 * convolution; in NCHW the direct convolution runs a simple kernel that F2
 * beats, so NCHW never gets DIRECT); F4 when its 64x64 row-streamed blocks,
 * (Cout/64) x (tiles/64), fill the device's compute units; F2 otherwise.
 *   layout: the activations' layout.
 *   algo:   host int32 out, one of wino_algo.
 * Errors: WINO_EINVAL (null algo, sizes < 0, channels < 1, unknown layout).
 */
typedef enum wino_algo { WINO_ALGO_DIRECT = 0, WINO_ALGO_F2 = 2, WINO_ALGO_F4 = 4 } wino_algo;
wino_status wino_select_algorithm(int32_t n, int32_t cin, int32_t cout, int32_t h, int32_t w,
                                  wino_layout layout, int32_t* algo);

/*
 * wino_f4_tap_kernel_choice -- the tap-GEMM kernel (WINO_TAP_ROWS, WINO_TAP_WAVES
 * or one of the WINO_TAP_RESIDENT_* shapes) that a SPLIT wino_f4_conv_int8 runs for an
 * n x h x w input, under the plan's wino_f4_plan_set_tap_kernel setting.
 * Host only, no device work.  kind: host int32 out.
 * Errors: WINO_EINVAL (null plan or kind, negative sizes), WINO_EUNSUPPORTED
 * (sizes beyond the library's limits).
 */
wino_status wino_f4_tap_kernel_choice(wino_f4_plan_t plan, int32_t n, int32_t h, int32_t w, int32_t* kind);

/*
 * wino_f2_plan, wino_f2_plan_tables -- the same offline step for Winograd
 * F(2x2, 3x3) (Sec. II: B^T, G = Gint / 2 and A^T of the F2 algorithm; the
 * tap-wise scheme of Sec. III with 16 taps, t = 4a + b).  Arguments, errors
 * and exactness as for the F4 functions, except that in_exp, w_exp, e_g and
 * sh have 16 entries and uq is [16][cin][cout].  The resulting plan runs 4x4
 * input tiles at stride 2 and 2x2 output tiles through the same execution
 * entry points (wino_f4_conv_int8 SPLIT and FUSED, wino_f4_workspace_bytes,
 * wino_f4_input_transform, wino_f4_tap_gemm, wino_f4_calibrate_output, the
 * debug exports and wino_f4_plan_info, whose table arguments then hold 16
 * entries).
 */
wino_status wino_f2_plan(wino_f4_plan_t* out, const float* w_oihw, int32_t cin, int32_t cout,
                         const int8_t* in_exp, const int8_t* w_exp, const int32_t* bias,
                         int32_t out_shift, int32_t relu, hipStream_t stream);
wino_status wino_f2_plan_tables(const float* w_oihw, int32_t cin, int32_t cout, const int8_t* in_exp,
                                const int8_t* w_exp, const int32_t* bias, int32_t out_shift, int8_t* e_g,
                                int8_t* sh, int32_t* e_o, int32_t* epilogue_bits, int8_t* uq);

/*
 * wino_f4_plan_device, wino_f2_plan_device -- the same plan with the weight
 * transform, the tap calibration and the tap-wise quantization (Sec. III-B:
 * U = G f G^T, e_G[t] the smallest e with max |U_t| <= 128 2^e, Uq =
 * clamp(R(U / 2^e_G))) computed on the GPU.  The paper transforms weights
 * inside the accelerator because Winograd-domain weights are four times the
 * spatial ones (Sec. IV); here the transform is a plan-time pass on the
 * device that writes Uq straight into the tap-GEMM layout.
 *   w_oihw_dev  device fp32 [cout][cin][3][3], contiguous, finite; read on
 *               `stream`, not retained.
 * Every other argument is the host argument of wino_f4_plan / wino_f2_plan.
 * Exact: the result is identical to wino_f4_plan / wino_f2_plan on the same
 * weights (every rounding and range decision is taken on an exact
 * floating-point expansion of d^2 U).  Allocates the plan's device memory
 * and a temporary; synchronizes `stream` before returning.  Errors as for
 * wino_f4_plan (WINO_EINVAL also for a NULL or non-finite weight tensor);
 * on error *out is NULL.  wino_f4_plan_info(uq) of such a plan reads Uq back
 * from the device.
 */
wino_status wino_f4_plan_device(wino_f4_plan_t* out, const float* w_oihw_dev, int32_t cin, int32_t cout,
                                const int8_t* in_exp, const int8_t* w_exp, const int32_t* bias,
                                int32_t out_shift, int32_t relu, hipStream_t stream);
wino_status wino_f2_plan_device(wino_f4_plan_t* out, const float* w_oihw_dev, int32_t cin, int32_t cout,
                                const int8_t* in_exp, const int8_t* w_exp, const int32_t* bias,
                                int32_t out_shift, int32_t relu, hipStream_t stream);

/*
 * wino_f4_plan_int8, wino_f2_plan_int8 -- plan from int8 spatial weights
 * f_hat = w_int8 * 2^w_scale_exp (the quantized weights that the tap-wise
 * formula of Sec. III transforms; one power-of-two scale per layer, e.g. from
 * direct_conv_quantize_weights after reordering to OIHW).  d^2 U = Gint w
 * Gint^T is then an integer, so the transform and the tap-wise quantization
 * run in integer arithmetic on the GPU.
 *   w_oihw_dev    device int8 [cout][cin][3][3], contiguous; read on `stream`.
 *   w_scale_exp   e_f in [-126, 120] (f_hat is then an exact fp32 value).
 * Other arguments and errors as for wino_f4_plan_device.  The result is
 * identical to wino_f4_plan / wino_f2_plan applied to the fp32 weights
 * w_int8 * 2^w_scale_exp.
 */
wino_status wino_f4_plan_int8(wino_f4_plan_t* out, const int8_t* w_oihw_dev, int32_t w_scale_exp, int32_t cin,
                              int32_t cout, const int8_t* in_exp, const int8_t* w_exp, const int32_t* bias,
                              int32_t out_shift, int32_t relu, hipStream_t stream);
wino_status wino_f2_plan_int8(wino_f4_plan_t* out, const int8_t* w_oihw_dev, int32_t w_scale_exp, int32_t cin,
                              int32_t cout, const int8_t* in_exp, const int8_t* w_exp, const int32_t* bias,
                              int32_t out_shift, int32_t relu, hipStream_t stream);

/*
 * wino_f4_plan_i10, wino_f2_plan_i10, wino_f4_plan_tables_i10,
 * wino_f2_plan_tables_i10 -- the int8/10 variant (Sec. V): int8 input and
 * output in the spatial domain, 10-bit integers in the Winograd domain.  Vq
 * and Uq are quantized to [-512, 511] with power-of-two tap scales chosen
 * from 2^9 (Eq. quant with n = 10: e_G[t] is the smallest e with
 * max |U_t| <= 512 2^e); everything else is the 8-bit scheme.  Arguments,
 * errors and exactness as for wino_f4_plan / wino_f4_plan_tables, except
 * that in_exp should come from wino_f4_calibrate_input_i10 and the tables'
 * uq output is int16 [ntap][cin][cout].  The resulting plan runs through
 * wino_f4_conv_int8 (SPLIT only; FUSED returns WINO_EUNSUPPORTED),
 * wino_f4_workspace_bytes (twice the 8-bit workspace: Vq is fp16),
 * wino_f4_input_transform, wino_f4_tap_gemm, wino_f4_calibrate_output and
 * the debug exports (wino_f4_debug_input_transform then writes fp16 values
 * [ntap][ntiles][cin], each an exact 10-bit integer).  wino_f4_plan_info
 * returns its exponents and epilogue width; its uq argument must be NULL
 * (WINO_EINVAL otherwise).  The tap GEMM runs on fp16 matrix cores: the
 * 10-bit integers are exact in fp16 and each 32-channel partial sum is an
 * integer below 2^24, exact in the fp32 accumulator, before it is added to
 * the int32 (or int64) accumulation -- the result is bit-exact.
 */
wino_status wino_f4_plan_i10(wino_f4_plan_t* out, const float* w_oihw, int32_t cin, int32_t cout,
                             const int8_t* in_exp, const int8_t* w_exp, const int32_t* bias, int32_t out_shift,
                             int32_t relu, hipStream_t stream);
wino_status wino_f2_plan_i10(wino_f4_plan_t* out, const float* w_oihw, int32_t cin, int32_t cout,
                             const int8_t* in_exp, const int8_t* w_exp, const int32_t* bias, int32_t out_shift,
                             int32_t relu, hipStream_t stream);
wino_status wino_f4_plan_tables_i10(const float* w_oihw, int32_t cin, int32_t cout, const int8_t* in_exp,
                                    const int8_t* w_exp, const int32_t* bias, int32_t out_shift, int8_t* e_g,
                                    int8_t* sh, int32_t* e_o, int32_t* epilogue_bits, int16_t* uq);
wino_status wino_f2_plan_tables_i10(const float* w_oihw, int32_t cin, int32_t cout, const int8_t* in_exp,
                                    const int8_t* w_exp, const int32_t* bias, int32_t out_shift, int8_t* e_g,
                                    int8_t* sh, int32_t* e_o, int32_t* epilogue_bits, int16_t* uq);

/* Releases a plan and its device memory.  NULL is ignored.  The caller must
 * ensure no convolution using the plan is still running. */
void wino_f4_plan_destroy(wino_f4_plan_t plan);

/*
 * wino_f4_plan_info -- the plan's tables, for inspection and parity tests.
 * Any output pointer may be NULL.  e_g, sh: host int8 [36]; e_o: host int32;
 * epilogue_bits: 32 or 64; uq: host int8 [36][cin][cout] (tap-major,
 * Uq[t][ci][co]); cin/cout: the plan's channel counts.  The last two outputs
 * extend the six-argument form: a caller holding only the handle (a plan made
 * on the device, or by another module) can size the uq buffer from them
 * before asking for it.
 */
wino_status wino_f4_plan_info(wino_f4_plan_t plan, int8_t* e_g, int8_t* sh, int32_t* e_o,
                              int32_t* epilogue_bits, int8_t* uq, int32_t* cin, int32_t* cout);

/*
 * Workspace bytes that wino_f4_conv_int8 needs for this plan, batch and image
 * size (SPLIT: the tap-major int8 Winograd-domain input, 36 x tiles x Cin
 * rounded up to the kernel's blocking, followed, when the plan forces the
 * stream-K split (WINO_TAP_ROWS_STREAMK) and the shape leaves a partial last
 * round of blocks, by that split's counters and partial sums: 512 KiB per
 * compute unit; FUSED: 0).  A SPLIT workspace of at least the Vq part but
 * smaller than this runs the same result without the split.  Returns 0 for
 * an invalid plan or negative sizes.
 */
size_t wino_f4_workspace_bytes(wino_f4_plan_t plan, int32_t n, int32_t h, int32_t w,
                               wino_variant variant);

/*
 * wino_f4_conv_int8 -- the online path (Sec. III scheme; operator dataflow
 * of Sec. IV-B2): input transform B^T d B of every 6x6 tile, tap-wise
 * requantization to int8 with 2^e_B[t], 36 int8 tap GEMMs with int32
 * accumulation, alignment by 2^sh[t], output transform A^T M A, bias,
 * requantization and optional ReLU.  Bit-exact integer arithmetic.
 *
 *   x          device int8 input, layout `layout`, [n][cin][h][w] or
 *              [n][h][w][cin]; not modified.
 *   y          device int8 output, same layout with cout channels; must not
 *              overlap x or the workspace.
 *   n, h, w    batch and image size, >= 0 (a zero size is a no-op), with
 *              n * ceil(h/4) * ceil(w/4) < 2^26 and each of h, w <= 65536.
 *   workspace  device memory of at least wino_f4_workspace_bytes() bytes
 *              (ignored for FUSED; may be NULL then); contents are scratch.
 *   stream     all work is enqueued on this stream; no host synchronization.
 * A plan may be used concurrently on several streams with separate
 * workspaces.  The device current at the call must be the one the plan was
 * made on (WINO_EINVAL otherwise; the same holds for every call below that
 * takes a plan and device data).  Errors: WINO_EINVAL, WINO_EUNSUPPORTED,
 * WINO_EWORKSPACE, WINO_EHIP (launch failure reported by hipGetLastError).
 */
wino_status wino_f4_conv_int8(wino_f4_plan_t plan, const int8_t* x, int8_t* y, int32_t n,
                              int32_t h, int32_t w, wino_layout layout, wino_variant variant,
                              void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * wino_f4_conv_int8_noalloc -- wino_f4_conv_int8 (SPLIT) for callers that
 * cannot allocate device memory: code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc.  It allocates nothing and takes no
 * workspace: the input-transform workspace is a file-scope device array of
 * WINO_NOALLOC_SCRATCH_BYTES (64 MiB) that each GPU the library runs on holds
 * until the process ends; its address is looked up once per device, on the
 * first call made with that device current.
 *
 *   plan, x, y, n, h, w, layout, stream: as for wino_f4_conv_int8.
 * Every call on one GPU shares that GPU's array and leaves its contents
 * behind (nothing in it needs clearing): calls that overlap on one GPU, e.g.
 * on two streams without ordering between them, race and must not be made.
 * It never splits the tap GEMM's last round (WINO_TAP_ROWS_STREAMK): the
 * array holds the input-transform workspace only.
 * Errors: as for wino_f4_conv_int8 (SPLIT), and WINO_EWORKSPACE when the
 * layer's input-transform workspace (36 x tiles x Cin, each rounded up to a
 * multiple of 64: wino_f4_workspace_bytes without a stream-K part) exceeds
 * WINO_NOALLOC_SCRATCH_BYTES (checked before any device work); WINO_EHIP if
 * the array's address cannot be obtained.
 */
#define WINO_NOALLOC_SCRATCH_BYTES (64u << 20)
wino_status wino_f4_conv_int8_noalloc(wino_f4_plan_t plan, const int8_t* x, int8_t* y, int32_t n,
                                      int32_t h, int32_t w, wino_layout layout, hipStream_t stream);

/*
 * The two launches of the SPLIT variant as separate calls, for callers that
 * schedule or time them individually; wino_f4_conv_int8(SPLIT) equals
 * wino_f4_input_transform followed by wino_f4_tap_gemm on the same stream.
 * wino_f4_input_transform: x -> workspace (Vq, the tap-major int8
 *   Winograd-domain input: B^T d B and the tap-wise requantization).
 * wino_f4_tap_gemm: workspace -> y (the 36 tap GEMMs, alignment, A^T M A,
 *   bias, requantization, ReLU, store).  `workspace` must hold the Vq
 *   written by wino_f4_input_transform for the same plan, n, h, w and
 *   workspace_bytes; the tap GEMM leaves Vq unchanged, so it may run again on
 *   it, and uses the part past Vq as scratch for a stream-K split (its
 *   counters, which the input transform zeroes and every split launch leaves
 *   at zero, and its partial sums).
 * Arguments, errors and stream semantics as for wino_f4_conv_int8.
 */
wino_status wino_f4_input_transform(wino_f4_plan_t plan, const int8_t* x, int32_t n, int32_t h, int32_t w,
                                    wino_layout layout, void* workspace, size_t workspace_bytes,
                                    hipStream_t stream);
wino_status wino_f4_tap_gemm(wino_f4_plan_t plan, void* workspace, size_t workspace_bytes, int8_t* y,
                             int32_t n, int32_t h, int32_t w, wino_layout layout, hipStream_t stream);

/*
 * wino_f4_calibrate_input -- max-abs calibration of the input tap scales
 * (Sec. III: x_max calibrated from observed maxima; power-of-two rule of
 * Sec. III-B).  Computes absmax[t] = max over all tiles and channels of
 * |(B^T d B)_t| on the GPU and e_B[t] = min(15, max(0, smallest e with
 * absmax[t] <= 128 * 2^e)).  Synchronizes `stream` before returning.
 *   x: device int8 input as for wino_f4_conv_int8.
 *   absmax: host int32 [36] or NULL;  e_b: host int8 [36] or NULL.
 * Allocates and frees a small device buffer (an offline step).
 */
wino_status wino_f4_calibrate_input(const int8_t* x, int32_t n, int32_t cin, int32_t h,
                                    int32_t w, wino_layout layout, int32_t* absmax,
                                    int8_t* e_b, hipStream_t stream);

/* wino_f2_calibrate_input -- the same for F(2x2, 3x3): 4x4 tiles at stride
 * 2, absmax and e_b with 16 entries. */
wino_status wino_f2_calibrate_input(const int8_t* x, int32_t n, int32_t cin, int32_t h,
                                    int32_t w, wino_layout layout, int32_t* absmax,
                                    int8_t* e_b, hipStream_t stream);

/* wino_f4_calibrate_input_i10, wino_f2_calibrate_input_i10 -- the input
 * calibration of the int8/10 variant (Sec. V): the same maxima, with
 * e_B[t] = min(15, max(0, smallest e with absmax[t] <= 512 * 2^e)) for
 * 10-bit input taps.  Arguments and errors as for wino_f4_calibrate_input
 * (36 or 16 entries). */
wino_status wino_f4_calibrate_input_i10(const int8_t* x, int32_t n, int32_t cin, int32_t h, int32_t w,
                                        wino_layout layout, int32_t* absmax, int8_t* e_b, hipStream_t stream);
wino_status wino_f2_calibrate_input_i10(const int8_t* x, int32_t n, int32_t cin, int32_t h, int32_t w,
                                        wino_layout layout, int32_t* absmax, int8_t* e_b, hipStream_t stream);

/*
 * wino_f4_calibrate_output -- max-abs calibration of the output shift: runs
 * the online path up to z = Y + bias and returns zmax = max |z| over all
 * in-image outputs and out_shift = min(62, max(0, smallest s with
 * zmax <= 128 * 2^s)).  The plan's own out_shift and relu are ignored.
 * Arguments as for wino_f4_conv_int8 (SPLIT workspace); zmax, out_shift are
 * host pointers (either may be NULL).  Synchronizes `stream`.
 */
wino_status wino_f4_calibrate_output(wino_f4_plan_t plan, const int8_t* x, int32_t n, int32_t h,
                                     int32_t w, wino_layout layout, void* workspace,
                                     size_t workspace_bytes, int64_t* zmax, int32_t* out_shift,
                                     hipStream_t stream);

/*
 * Stage exports for parity tests (not on the hot path).
 * wino_f4_debug_input_transform: the int8 tap-major Winograd-domain input
 *   Vq[t][tile][ci] (tile = (img*ceil(h/4) + ty)*ceil(w/4) + tx), written to
 *   device int8 `vq` of 36 * tiles * cin bytes.
 * wino_f4_debug_tap_gemm: the raw int32 tap GEMM results M[t][tile][co]
 *   (before alignment), written to device int32 `m` of 36 * tiles * cout
 *   elements.
 * Both need the SPLIT workspace and run on `stream` without synchronizing.
 */
wino_status wino_f4_debug_input_transform(wino_f4_plan_t plan, const int8_t* x, int32_t n,
                                          int32_t h, int32_t w, wino_layout layout, int8_t* vq,
                                          void* workspace, size_t workspace_bytes,
                                          hipStream_t stream);
wino_status wino_f4_debug_tap_gemm(wino_f4_plan_t plan, const int8_t* x, int32_t n, int32_t h,
                                   int32_t w, wino_layout layout, int32_t* m, void* workspace,
                                   size_t workspace_bytes, hipStream_t stream);

/*
 * direct_conv_quantize_weights -- spatial int8 weights for the direct
 * baseline: one power-of-two scale per layer, e = smallest e with
 * max |f| <= 128 * 2^e, w = clamp(R(f / 2^e), -128, 127) (Eq. quant with the
 * power-of-two rule).  w_oihw: host fp32 [cout][cin][3][3]; w_ohwi: host int8
 * [cout][3][3][cin] (output); e: host int32 (output).  Exact arithmetic.
 */
wino_status direct_conv_quantize_weights(const float* w_oihw, int32_t cout, int32_t cin,
                                         int8_t* w_ohwi, int32_t* e);

/*
 * direct_conv_int8 -- the standard (im2col-style) 3x3 convolution the paper
 * compares against (Sec. IV-A, im2col engine; Sec. V), as an implicit GEMM
 * on int8 MFMA: z = sum x * w + bias (exact int32), out = clamp(R(z /
 * 2^out_shift), -128, 127), optional ReLU.  Same geometry and layouts as
 * wino_f4_conv_int8.
 *   w_ohwi  device int8 [cout][3][3][cin];  bias: device int32 [cout] or NULL.
 *           OHWI rather than OIHW: the implicit GEMM's reduction index is
 *           (ky, kx, ci), so each output channel's 9*cin weights are one
 *           contiguous row that the kernel streams in 16-byte pieces next to
 *           NHWC pixels.  direct_conv_quantize_weights writes this order from
 *           fp32 OIHW; an OIHW int8 tensor becomes it by a permute (0, 2, 3, 1).
 *   1 <= cin <= 8192 (keeps the int32 accumulator exact), 1 <= cout <= 65536,
 *   out_shift in [0, 31], relu 0|1.  Asynchronous on `stream`.
 */
wino_status direct_conv_int8(const int8_t* x, const int8_t* w_ohwi, const int32_t* bias, int8_t* y,
                             int32_t n, int32_t cin, int32_t cout, int32_t h, int32_t w,
                             wino_layout layout, int32_t out_shift, int32_t relu,
                             hipStream_t stream);

/*
 * wino_f4_conv_float -- the unquantized Winograd F(4x4, 3x3) convolution of
 * Eq. (winograd), Sec. II, evaluated in fp32: V = B^T d B, U = G f G^T,
 * M = sum_ci V (.) U, Y = A^T M A, every intermediate an fp32 value, no
 * tap-wise quantization, no bias, no requantization.  It is the real-valued
 * convolution the integer pipeline approximates, kept as a reference stage
 * whose floating-point intermediates a test can hold to a relative
 * tolerance; it is not on the hot path.
 *   x       device int8, NCHW [n][cin][h][w] or NHWC [n][h][w][cin]
 *   w_oihw  device fp32 [cout][cin][3][3]
 *   y       device fp32, same layout as x with cout channels (written)
 * 3x3, stride 1, pad 1; 1 <= cin, cout <= 65536; h, w <= 65536.  Empty
 * inputs launch nothing.  Asynchronous on `stream`; WINO_EINVAL for NULL
 * pointers or bad sizes, WINO_EUNSUPPORTED beyond the limits, WINO_EHIP if
 * the launch fails.
 */
wino_status wino_f4_conv_float(const int8_t* x, const float* w_oihw, float* y, int32_t n,
                               int32_t cin, int32_t cout, int32_t h, int32_t w,
                               wino_layout layout, hipStream_t stream);

/* Static description of a status code; never NULL. */
const char* wino_strerror(wino_status status);

#ifdef __cplusplus
}
#endif

#endif /* WINOF4_H */
