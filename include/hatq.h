/*
 * hatq.h -- C ABI of the MI355X (gfx950) Hadamard-domain INT8 linear operator.
 *
 * The operator is the inference-time layer of HaTQ ("Hadamard-Domain Model
 * Quantization for Learned Image Coding"): a convolution or fully connected
 * layer Y = X W^T + b (Eq. supp_linear_operator) evaluated with INT8 operands in
 * a Hadamard domain, in one of two per-layer forms (Sec. IV-B):
 *
 *   DH (double-Hadamard, Eq. double_hadamard_quantization): activations and
 *      weights are both transformed along the contracted input channels,
 *      Y = Q(X T_in) Q(W T_in)^T.
 *   WH (weight-only Hadamard, Eq. weight_only_hadamard_quantization): weights
 *      are transformed along output channels, activations are quantized in the
 *      original domain, and the accumulator is mapped back,
 *      Y = [Q(X) Q(T_out^T W)^T + b~] T_out^T   (Eq. supp_padded_wh).
 *
 * Transforms are block diagonal, B_C = I_{C/b} (x) H~_b, with H~_b the
 * unnormalized Sylvester matrix of order b (Eq. supp_sylvester, natural order).
 * The normalization 1/sqrt(b) of each side is folded into the dequantization
 * scale as one exact factor 1/b (Supplementary, "Deployment Realization").
 *
 * Quantization is symmetric INT8 with codes in [-127, 127] (Eq. symmetric_q):
 * per-sample dynamic activation scale s_x = ||S||_inf / 127 (Eq. current_scale)
 * and per-output-channel weight scale; rounding is round-half-to-even and x/s is
 * an IEEE fp32 division.  The INT8 x INT8 products accumulate in INT32
 * (Eq. integer_accumulation); the accumulator of channel c has scale
 * s_x * s_w,c (Eq. accumulator_scale).
 *
 * Conventions for every entry point:
 *  - Tensors are NHWC, row-major, densely packed.  All tensor pointers are
 *    DEVICE pointers owned by the caller (hatq_export_weights also takes host
 *    destinations); the library never allocates, frees or synchronizes, and
 *    keeps no global state.  Calls are reentrant; calls on one stream execute
 *    in order.
 *  - `stream` is a hipStream_t (NULL = the default stream).  Some launch
 *    shapes (the persistent convolution grids) follow the CU count of the
 *    current device; results do not depend on them.
 *  - Arguments are validated on the host before any launch.  On error nothing
 *    is launched and outputs are untouched.  A launch failure is reported as
 *    HATQ_EHIP; faults inside kernels surface at the caller's next
 *    synchronization.  Nothing is printed and no C++ exception crosses the ABI.
 *  - Unless noted, no entry point reads device memory on the host.
 */
#ifndef HATQ_H
#define HATQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    HATQ_OK = 0,
    HATQ_EINVAL = 1,        /* bad argument: null pointer, bad size, form mismatch */
    HATQ_EUNSUPPORTED = 2,  /* valid operator outside the kernels' supported geometry */
    HATQ_EWORKSPACE = 3,    /* caller-provided buffer too small */
    HATQ_EHIP = 4           /* a HIP launch or runtime call failed */
} hatq_status;

typedef enum { HATQ_DH = 0, HATQ_WH = 1 } hatq_form;

typedef enum {
    HATQ_OUT_I32 = 0,       /* raw INT32 accumulators [n][ho][wo][cout_pad], no bias;
                               WH accumulators stay in the output Hadamard basis */
    HATQ_OUT_F32 = 1,       /* dequantized fp32 output [n][ho][wo][cout], original basis */
    HATQ_OUT_I8 = 2         /* the next operand's INT8 codes [n][ho][wo][cout] (requantization,
                               Eq. integer_requantization) */
} hatq_out_mode;

/* Flags of the convolution entry points (bitwise or; 0 = none).
 *   HATQ_PAIRED: a WH layer whose next operand uses the same transform blocks
 *     (next_hblock == hblock > 1) with nothing applied between the layers
 *     (identity nonlinearity) may take the next operand through the cancellation
 *     of Table I: B_next y = B_next (B_Cout z) / b = z, z the dequantized
 *     accumulators before the output restore (Sylvester blocks square to b I).
 *     Neither butterfly then runs: the next operand's absmax is max|z|, its
 *     codes are those of z, and the integer transition uses B_next B_Cout = b I.
 *     Without the flag both transforms run explicitly (the general Table I
 *     transition, which a nonlinearity between the layers needs).  Ignored for
 *     every other layer and output. */
/*   HATQ_XQ_C64: the input codes xq are in the chunk-major layout
 *     [n][cin_pad/64][h][w][64] (64-channel planes) instead of [n][h][w][cin_pad],
 *     as hatq_fwht_quant_act_c64 and HATQ_YQ_C64 write them.  Same codes, same
 *     results; the window refills of the 5x5 stride-2 kernel then read whole
 *     128-byte lines (Eq. linear_operator: the contraction is unchanged, only
 *     where each code sits).  Supported for regular (not transposed) 5x5 stride-2
 *     layers with cin_pad % 64 == 0 and cout_pad 192 or 320, except a call
 *     whose epilogue transforms by the order 320 (a WH restore of order 320 or
 *     next_hblock 320 with a float or code output); HATQ_EUNSUPPORTED
 *     otherwise.
 *   HATQ_YQ_C64: code outputs (HATQ_OUT_I8, hatq_conv_int8_requant,
 *     hatq_conv_int8_int_transition) go out chunk-major,
 *     [n][cout/64][ho][wo][64]; needs cout % 64 == 0 (HATQ_EUNSUPPORTED
 *     otherwise), HATQ_EINVAL for F32 and I32 outputs. */
typedef enum { HATQ_PAIRED = 1, HATQ_XQ_C64 = 2, HATQ_YQ_C64 = 4 } hatq_conv_flags;

/* One layer's geometry.  Square kernels only.
 *   conv:        ho = (h + 2*pad - k)/stride + 1
 *   transposed:  ho = (h - 1)*stride - 2*pad + k + out_pad
 * hblock: block order b of the transform B = I (x) H_b; it acts on cin for DH
 * and on cout for WH.  b = 1 means no transform.  A power of two in [1, 128]
 * (Sylvester H~_b), or one of the orders m(C) of Eq. hadamard_order that the
 * Sylvester family lacks, built as Kronecker products with a Paley-I factor
 * (supplementary, Hadamard construction): 192 = P_12 (x) H~_16 and
 * 320 = P_20 (x) H~_16, index a*16 + l (Paley index a, Sylvester index l).
 * Those two are supported for DH layers in hatq_fwht_quant_act,
 * hatq_prepare_weights, hatq_conv_int8 and hatq_layer_forward (the DH
 * dequantization factor is fl(s_x s_w / b)), and by the activation-side
 * profiling and affine entry points (hatq_range_expansion,
 * hatq_fwht_quant_act_affine) for whole blocks (c % b == 0); the entry points
 * below that say so take them also for the convolution epilogues (192 with
 * cout_pad 192, 320 with cout_pad 320 and cin_pad % 64 == 0). */
typedef struct {
    int32_t cin, cout;
    int32_t k;
    int32_t stride, pad, out_pad;
    int32_t transposed;     /* 0: convolution, 1: transposed convolution */
    int32_t hblock;
} hatq_conv_desc;

/* Prepared weights: a plain view into the caller's device buffer, filled by
 * hatq_prepare_weights.  Layout of wq: [cout_pad][k_stride] int8, row co holds
 * the contraction index d = (kh*k + kw)*cin_pad + ci (the Kronecker order
 * I_{KhKw} (x) H of Eq. input_hadamard_transform); bytes d >= k_total are 0.
 * For a transposed convolution (kh, kw) index the kernel as stored in PyTorch
 * (weight[ci][co][kh][kw]).  w_scale and bias are fp32 [cout_pad]; for WH the
 * bias is the transformed b~ = B_Cout [b; 0] (Eq. supp_padded_wh_parameters).
 * wpack holds the same codes again in the order the convolution kernels stream
 * them (K-blocked: [pack_stride/64][cout_pad][64], contiguous per 64-deep
 * contraction step); it is library-internal and callers must not depend on
 * its order.  hatq_prepare_weights fills both copies. */
typedef struct {
    hatq_conv_desc d;
    int32_t form;           /* hatq_form, fixed for the layer's lifetime (Sec. IV-C) */
    int32_t cin_pad;        /* cin (DH: rounded up to hblock) */
    int32_t cout_pad;       /* cout (WH: rounded up to hblock) */
    int32_t k_total;        /* k*k*cin_pad */
    int32_t k_stride;       /* k_total rounded up to 64 */
    int8_t *wq;
    float *w_scale;
    float *bias;
    int8_t *wpack;          /* kernel-order copy of wq (see above) */
    int32_t pack_stride;    /* contraction bytes per output channel in wpack */
} hatq_weights;

/* Static description of a status code.  Never NULL. */
const char *hatq_status_string(int32_t status);

/* Output spatial size of `d` for an input of h x w.  HATQ_EINVAL if the result
 * would be empty. Host only. */
int32_t hatq_conv_out_hw(const hatq_conv_desc *d, int32_t h, int32_t w, int32_t *ho, int32_t *wo);

/* Bytes of device memory hatq_prepare_weights needs for `d` in form `form`
 * (0 for an invalid descriptor). */
size_t hatq_weights_bytes(const hatq_conv_desc *d, int32_t form);

/* Offline weight preparation (Eq. hadamard_linear_equivalence and
 * Eq. weight_only_hadamard_equivalence with the padded forms of the
 * supplementary; per-channel symmetric quantization, Eq. symmetric_q).
 *   w:    device fp32 weights in PyTorch layout, OIHW [cout][cin][k][k] for a
 *         convolution, IOHW [cin][cout][k][k] for a transposed convolution.
 *   bias: device fp32 [cout], or NULL for no bias.
 *   dst:  device buffer of at least hatq_weights_bytes(d, form) bytes; it holds
 *         wq, w_scale and bias afterwards.  `out` (host struct) receives the
 *         view into it.
 * The transform is evaluated in fp64 and rounded once to fp32; then
 * s_w,c = fl32(max|W'_c| / 127) (1 for an all-zero row) and
 * wq = clamp(rne(fl32(W'/s_w,c)), -127, 127).  Runs on `stream`.
 * Supported: DH needs cin % hblock == 0, WH needs cout % hblock == 0. */
int32_t hatq_prepare_weights(const hatq_conv_desc *d, int32_t form, const float *w,
                             const float *bias, void *dst, size_t dst_bytes,
                             hatq_weights *out, void *stream);

/* Copy prepared weights out in their documented layout (Eq. hadamard_linear_equivalence
 * and Eq. weight_only_hadamard_equivalence: the transformed, quantized operator):
 *   wq:      int8 [cout_pad][k][k][cin_pad], the codes of W' (row co holds
 *            d = (kh*k + kw)*cin_pad + ci, as W->wq without its zero K padding);
 *   w_scale: fp32 [cout_pad], s_w,c;  bias: fp32 [cout_pad] (WH: b~ = B_Cout [b; 0]).
 * Destinations may be host or device memory (any of them NULL to skip it); the
 * copies are enqueued on `stream` and host destinations hold the data once the
 * caller has synchronized the stream (with pageable host memory the HIP runtime
 * may complete the copy before returning). */
int32_t hatq_export_weights(const hatq_weights *W, int8_t *wq, float *w_scale, float *bias, void *stream);

/* Rebuild W->wpack from the codes in W->wq, for callers that write codes into
 * wq themselves (codes quantized elsewhere, e.g. loaded from a deployment
 * checkpoint, with w_scale and bias filled to match).  W must be a view returned
 * by hatq_prepare_weights (same geometry); wq bytes past k_total must be 0.
 * Runs on `stream`. */
int32_t hatq_pack_weights(const hatq_weights *W, void *stream);

/* Workspace bytes hatq_fwht_quant_act needs for a batch of n samples. */
size_t hatq_fwht_quant_ws_bytes(int32_t n);

/* Activation transform and quantization, steps a2-a4 of one layer
 * (Eq. input_hadamard_transform, Eq. symmetric_q, Eq. current_scale):
 *   S[p] = B_c x[p] along channels (hblock = 1: S = x),
 *   s_x[i] = fl32(max |S over sample i| / 127)  (1 if that max is 0),
 *   xq = clamp(rne(fl32(S / s_x[i])), -127, 127).
 *   x:        device fp32 [n][h][w][c].
 *   absmax:   NULL, or device fp32 [n] holding max |S| per sample already (as
 *             produced by hatq_conv_int8's next_absmax); then the input is read
 *             once instead of twice.
 *   xq:       device int8 [n][h][w][c].
 *   act_scale: device fp32 [n], receives s_x (unnormalized-domain scale).
 *   ws:       device workspace of hatq_fwht_quant_ws_bytes(n) bytes (unused
 *             when absmax is given).
 * Supported: c % hblock == 0, and c % 4 == 0 or hblock == 1; for the Kronecker
 * orders 192 and 320, h*w*c % 4 == 0. */
int32_t hatq_fwht_quant_act(const float *x, int32_t n, int32_t h, int32_t w, int32_t c,
                            int32_t hblock, const float *absmax, int8_t *xq, float *act_scale,
                            void *ws, size_t ws_bytes, void *stream);

/* hatq_fwht_quant_act with the codes in the chunk-major layout of HATQ_XQ_C64:
 *   xq: device int8 [n][c/64][h][w][64], 16-byte aligned; the code of channel
 *       64m + j of pixel p at ((i*(c/64) + m)*h*w + p)*64 + j for sample i.
 * Same codes and scales as hatq_fwht_quant_act.  Supported: c % 64 == 0 and
 * hblock a power of two at most 64 (HATQ_EUNSUPPORTED otherwise). */
int32_t hatq_fwht_quant_act_c64(const float *x, int32_t n, int32_t h, int32_t w, int32_t c,
                                int32_t hblock, const float *absmax, int8_t *xq, float *act_scale,
                                void *ws, size_t ws_bytes, void *stream);

/* hatq_fwht_quant_act without a workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid allocation): the two-pass form (absmax, then codes) keeps the
 * per-sample absmax in a static array inside the library, one copy per GPU,
 * of HATQ_NOALLOC_MAX_SAMPLES x 32 floats (512 KB: the per-block maxima of a
 * sample spread over 32 slots), held until the process ends.
 * Arguments, results and support as hatq_fwht_quant_act with absmax = NULL;
 * n > HATQ_NOALLOC_MAX_SAMPLES returns HATQ_EUNSUPPORTED.  Allocates nothing.
 * Every call on one GPU shares that GPU's array (it is cleared by the call
 * itself on the stream), so calls that overlap on one GPU (on different
 * streams, or from several threads) race and must not be issued. */
#define HATQ_NOALLOC_MAX_SAMPLES 4096
int32_t hatq_fwht_quant_act_noalloc(const float *x, int32_t n, int32_t h, int32_t w, int32_t c, int32_t hblock,
                                    int8_t *xq, float *act_scale, void *stream);

/* INT8 convolution with INT32 accumulation and the fused epilogue, steps a5-a6
 * (Eq. integer_accumulation, Eq. accumulator_scale, Table I).
 *   xq:        device int8 [n][h][w][cin_pad] (codes from hatq_fwht_quant_act).
 *   act_scale: device fp32 [n].
 *   mode HATQ_OUT_I32: y is int32 [n][ho][wo][cout_pad], raw accumulators.
 *   mode HATQ_OUT_F32: y is fp32 [n][ho][wo][cout]:
 *     DH: y = fma(float(acc), fl(s_x*s_w,c) * (1/b), bias_c);
 *     WH: z_c = fma(float(acc), fl(s_x*s_w,c), b~_c) (scale before the basis
 *         change, Supplementary "General Nonlinearities"), y = (B_Cout z)/b,
 *         truncated to cout.
 *   mode HATQ_OUT_I8: y is int8 [n][ho][wo][cout], the next layer's codes
 *     clamp(rne(fl32(y' / s))), y' = B_next y with blocks of next_hblock (1: y'
 *     = y) and s = out_scale[n], a static per-sample scale (Eq.
 *     integer_requantization); exactly hatq_conv_int8_requant with that static
 *     scale.  y (fp32) itself is never written.
 *   out_scale: device fp32 [n], required in I8 mode, NULL otherwise.
 *   next_hblock / next_absmax (F32 mode only): if next_absmax is non-NULL it
 *     receives, per sample, max |B_{next} y| with block size next_hblock (1: max
 *     |y|), the exact value hatq_fwht_quant_act would compute from y; the next
 *     layer can then quantize y reading it once.  It is overwritten, not
 *     accumulated.  y may be NULL in F32 mode when next_absmax is given: the
 *     call then only produces next_absmax (the first pass of
 *     hatq_conv_int8_requant's dynamic scale).  With HATQ_PAIRED (see above)
 *     a WH layer whose block equals next_hblock takes max |z| instead.
 *   next_hblock (I8 mode): the next operand's transform block.
 *   flags:     HATQ_PAIRED, HATQ_XQ_C64, HATQ_YQ_C64 (I8 mode only), or 0.
 * Supported: cin_pad % 64 == 0 with k <= 8, or cin_pad <= 4 with k*k*cin_pad <= 128;
 * cout_pad % 64 == 0; WH block and next_hblock a power of two at most 64, or
 * a Kronecker order equal to cout_pad: 192 (P_12 (x) H~_16), or 320
 * (P_20 (x) H~_16) when cin_pad % 64 == 0 (applied as H~_16 then the Paley
 * factor; the WH restore multiplies by B^T), or 128 with cout_pad 128 or 256
 * (with cin_pad <= 4 only for the row-run geometry: k <= 8, stride <= 2,
 * k*cin_pad <= 16, not transposed) (I8: as hatq_conv_int8_requant).  Transposed: stride 2.  xq and y (F32, I32) must be
 * 16-byte aligned, y in I8 mode 4-byte aligned. */
int32_t hatq_conv_int8(const hatq_weights *W, const int8_t *xq, const float *act_scale,
                       int32_t n, int32_t h, int32_t w, int32_t out_mode, const float *out_scale, void *y,
                       int32_t next_hblock, float *next_absmax, int32_t flags, void *stream);

/* INT8 convolution with the requantizing epilogue (step a6, I8 output; Eq.
 * integer_requantization with the dynamic per-tensor scale of Eq. symmetric_q):
 * the layer's fp32 output y (as hatq_conv_int8 computes it in F32 mode) is
 * transformed for the next layer, y' = B_next y with blocks of next_hblock (1:
 * y' = y, the WH input case), and quantized in registers,
 *   yq = clamp(rne(fl(y' / s)), -127, 127),
 * exactly as hatq_fwht_quant_act(y, ..., next_hblock, absmax = next_absmax)
 * would from y (the same fp32 butterflies in the same order, the same
 * rounding); y itself is never written.  With HATQ_PAIRED a WH layer whose
 * block equals next_hblock quantizes z instead (B_next y = z in exact
 * arithmetic, Table I): the codes are those of z, and can differ from the
 * explicit path's by the rounding of its two fp32 butterflies.
 *   next_absmax: device fp32 [n] with max |B_next y| per sample (from an
 *     earlier hatq_conv_int8 call with y = NULL, or an upper bound of it); the
 *     scale is then s = fl32(next_absmax / 127) (1 if it is 0) and is written to
 *     next_scale.  NULL: next_scale [n] is an input, a static scale.
 *   next_scale: device fp32 [n], the next layer's act_scale.
 *   yq:        device int8 [n][ho][wo][cout], the next layer's xq (with
 *              HATQ_YQ_C64: [n][cout/64][ho][wo][64]).
 *   flags:     HATQ_PAIRED, HATQ_XQ_C64, HATQ_YQ_C64, or 0.
 * Supported: as hatq_conv_int8, with cout % 4 == 0 and cout % next_hblock == 0. */
int32_t hatq_conv_int8_requant(const hatq_weights *W, const int8_t *xq, const float *act_scale,
                               int32_t n, int32_t h, int32_t w, int32_t next_hblock,
                               const float *next_absmax, float *next_scale, int8_t *yq,
                               int32_t flags, void *stream);

/* Affine activation quantization (Eq. affine_q, Eq. uniform_q), the dynamic
 * per-sample form of the paper's PTQ setting, on the signed grid [-128, 127]
 * (the paper's unsigned grid shifted by -128: the same dequantized values, codes
 * that the signed INT8 product takes).  For S = the activation transform of
 * each sample (as hatq_fwht_quant_act): with lo = max(-min S, 0), hi = max(max
 * S, 0), r = fl32(hi + lo):
 *   s = fl32(r / 255), z = clamp(rne(fl32(lo / s)) - 128, -128, 127); r = 0 gives
 *   s = 1, z = 0;  xq = clamp(rne(fl32(S / s)) + z, -128, 127).
 *   act_scale, act_zero: device fp32 / int32 [n], written.
 *   ws: device workspace of hatq_fwht_quant_affine_ws_bytes(n) bytes.
 * hblock: a power of two <= 128 or a Kronecker order (192, 320).
 * Supported: c % hblock == 0, h*w*c % 4 == 0, n <= 65535. */
size_t hatq_fwht_quant_affine_ws_bytes(int32_t n);
int32_t hatq_fwht_quant_act_affine(const float *x, int32_t n, int32_t h, int32_t w, int32_t c, int32_t hblock,
                                   int8_t *xq, float *act_scale, int32_t *act_zero, void *ws, size_t ws_bytes,
                                   void *stream);

/* Weight sums for the zero-point correction: tapsum[t][c] = sum over ci of the
 * code W_q[c][t][ci] for each tap t < k*k, then tapsum[k*k][c] = their total.
 * hatq_tapsum_len gives the int32 entries ((k*k + 1) * cout_pad, 0 for invalid
 * weights); tapsum is device memory, 16-byte aligned, written on the stream. */
size_t hatq_tapsum_len(const hatq_weights *W);
int32_t hatq_weight_tapsums(const hatq_weights *W, int32_t *tapsum, void *stream);

/* INT8 convolution of affine codes (Eq. integer_accumulation with zero points
 * z_x per sample and z_w = 0): the accumulator is the sum of (x - z_x) w over
 * the input pixels inside the image (padding is the value zero), formed as the
 * sum of x w minus z_x times the weight sum of the pixel's inside taps; then
 * the same output modes as hatq_conv_int8 (HATQ_OUT_I32: these centered
 * accumulators; HATQ_OUT_F32: the same epilogue with s_x = act_scale).
 *   act_zero: device int32 [n] (from hatq_fwht_quant_act_affine).
 *   tapsum:   from hatq_weight_tapsums for W.
 * Supported: as hatq_conv_int8 (no next-operand absmax; not a WH layer of
 * block 128). */
int32_t hatq_conv_int8_affine(const hatq_weights *W, const int8_t *xq, const float *act_scale,
                              const int32_t *act_zero, const int32_t *tapsum, int32_t n, int32_t h, int32_t w,
                              int32_t out_mode, void *y, void *stream);

/* Integer-only transition (Eq. integer_accumulation, Eq.
 * integer_fixed_point_scale, Eq. integer_hadamard_transition, the integer
 * column of Table I) with static per-tensor scales: the layer's INT32
 * accumulators become the next layer's INT8 codes with no floating point.
 *
 * hatq_int_table_len: int32 entries of the parameter table of W (2*cout_pad + 1),
 * 0 for invalid weights.
 *
 * hatq_int_transition_params: calibration step, fills the table on the device.
 *   s_x:   the static scale of W's input codes (unnormalized domain).
 *   s_y:   the static scale of the next operand's codes.
 *   next_hblock: the next operand's transform block (1: none), a power of two
 *          <= 64, 192 or 320 (not 128, and W not a WH layer of block 128:
 *          HATQ_EUNSUPPORTED); the overflow bound depends on it, so the table serves
 *          only calls with this next_hblock.
 *   table: device int32 [2*cout_pad + 1], 16-byte aligned, written as
 *     M[c]         = rne(2^n rho_c), rho_c = u_c / (beta_out s_y),
 *     b_int[c]     = rne(b_c / u_c),  u_c = s_x s_w,c / beta_in,
 *     table[2*cout_pad] = n,
 *   with (beta_in, beta_out) = (hblock, 1) for DH and (1, hblock) for WH (one
 *   accumulator step is worth u_c; the WH output transform divides by its
 *   block), b the prepared bias (WH: in the output basis) and n the largest
 *   shift in [0, 62] with every M_c <= floor(2^62 / (A_max G)) and < 2^31,
 *   A_max = k*k*cin_pad*127^2 + max|b_int|, G = (WH: hblock) * next_hblock:
 *   every int64 sum of the transition is then exact.  fp64 arithmetic with
 *   correctly rounded division.
 *   Enqueued on `stream` like every other call (it does not wait): when no
 *   shift fits (or |b_int| >= 2^30) the table holds n = -1 and every M_c = 0,
 *   which the caller reads back after its own synchronization; a transition
 *   with such a table writes all-zero codes.
 *
 * hatq_conv_int8_int_transition: convolution plus the integer epilogue,
 *   p = M (.) (acc + b_int) in int64, v = B_Cout^T p (WH; truncated to cout),
 *   w = B_next v (blocks of next_hblock), yq = clamp(rne(w / 2^n), -127, 127)
 *   with rne rounding exact halves to even; no act_scale (it is inside M).
 *   table: as written by hatq_int_transition_params for W and next_hblock.
 *   yq:    device int8 [n][ho][wo][cout], the next layer's codes.
 *   flags: HATQ_PAIRED (a WH layer whose block equals next_hblock then uses
 *          B_next B_Cout = b I: bit-identical codes, no butterflies),
 *          HATQ_XQ_C64, HATQ_YQ_C64, or 0.
 *   Supported: as hatq_conv_int8_requant. */
size_t hatq_int_table_len(const hatq_weights *W);
int32_t hatq_int_transition_params(const hatq_weights *W, float s_x, float s_y, int32_t next_hblock,
                                   int32_t *table, void *stream);
int32_t hatq_conv_int8_int_transition(const hatq_weights *W, const int8_t *xq, int32_t n, int32_t h,
                                      int32_t w, int32_t next_hblock, const int32_t *table,
                                      int8_t *yq, int32_t flags, void *stream);

/* Range-expansion profiling (Eq. hadamard_sensitivity): for each sample k of
 * a layer's input x, whether the layer's input-side transform enlarges the
 * range, ||H x_k||_inf > ||x_k||_inf with H = B_C / sqrt(hblock) orthonormal
 * (B_C the block-diagonal Sylvester transform, channels zero-padded to a
 * multiple of hblock).  Decided exactly as max|S|^2 > hblock * max|x|^2 in
 * fp64, S the fp32 butterfly transform hatq_fwht_quant_act applies.
 *   x:      device fp32 [n][h][w][c], 16-byte aligned; n <= 65535.
 *   hblock: a supported order (1: no transform, never an expansion); the
 *           Kronecker orders 192 and 320 need c % hblock == 0 and h*w*c % 4 == 0.
 *   amax:   device fp32 [2n], written: max|x_k| at [k], max|S_k| at [n + k].
 *   flags:  NULL, or device int32 [n] receiving 1 (expands) or 0.
 *   count:  NULL, or device int32 [1] to which the number of expanding samples
 *           is added (not overwritten: calls over the batches of a profiling
 *           set accumulate).
 * The probability p_l is *count / images over the profiling set. */
int32_t hatq_range_expansion(const float *x, int32_t n, int32_t h, int32_t w, int32_t c, int32_t hblock,
                             float *amax, int32_t *flags, int32_t *count, void *stream);

/* Form rule (Eq. layerwise_hadamard_selection): *form = HATQ_WH if
 * p = expansions / images (correctly rounded fp64) exceeds tau, else HATQ_DH.
 * HATQ_EINVAL for images <= 0, expansions outside [0, images] or a non-finite
 * tau.  Host only. */
int32_t hatq_select_form(int64_t expansions, int64_t images, double tau, int32_t *form);

/* Transform order rule (Eq. hadamard_order with the supplementary Hadamard
 * construction): m(c) = the smallest order m >= 4 ceil(c/4) for which a
 * Hadamard matrix is built, the orders being 1 and 2, q + 1 (Paley-I, q an odd
 * prime power, q = 3 mod 4), 2(q + 1) (Paley-II, q = 1 mod 4), and every
 * product of two of them (Kronecker products); m(192) = 192 and m(320) = 320.
 * Returns m(c), or 0 for c < 1 or c > 4096.  Whether the kernels take the
 * order is a separate question: hblock documents that (the powers of two up to
 * 128, 192 and 320).  Host only. */
int32_t hatq_hadamard_order(int32_t c);

/* Workspace bytes of hatq_layer_forward for an input of n x h x w. */
size_t hatq_layer_ws_bytes(const hatq_weights *W, int32_t n, int32_t h, int32_t w);

/* One whole layer (step a7): hatq_fwht_quant_act then hatq_conv_int8 in F32
 * mode, with the transform of the layer's own form (DH: hblock on cin; WH: none
 * on the activations).
 *   form:      must equal W->form (the per-layer form flag), else HATQ_EINVAL.
 *   x:         device fp32 [n][h][w][cin].
 *   x_absmax:  NULL, or per-sample max |T_in x| already known (see above).
 *   y:         device fp32 [n][ho][wo][cout].
 *   act_scale: NULL, or device fp32 [n] receiving s_x.
 *   next_hblock, next_absmax: as in hatq_conv_int8.
 *   ws:        at least hatq_layer_ws_bytes(W, n, h, w) bytes of device memory. */
int32_t hatq_layer_forward(const hatq_weights *W, int32_t form, const float *x, int32_t n,
                           int32_t h, int32_t w, const float *x_absmax, float *y,
                           float *act_scale, int32_t next_hblock, float *next_absmax,
                           void *ws, size_t ws_bytes, void *stream);

#ifdef __cplusplus
}
#endif
#endif /* HATQ_H */
