/*
 * mxconv.h -- quantize-once MX convolution on MI355X (gfx950).
 *
 * The hot path of MicroQonv: each convolution tensor (activations X, weights
 * W, output gradients G_Y) is quantized exactly once into an OCP-MX format
 * whose shared E8M0 scale covers a square block spanning both directions in
 * which the tensor is contracted (Sec. IV-B); activations are quantized
 * before a channel-batch-first im2col (Sec. IV-A), which then only moves
 * codes; the three convolution GEMMs of Sec. II-C / Sec. IV-B (forward,
 * input gradient, weight gradient) consume the MX codes directly on the
 * block-scaled matrix cores.
 *
 * ---------------------------------------------------------------------------
 * Formats
 *   MXC_E4M3: FP8 E4M3 elements (OCP "E4M3FN": bias 7, max 448, no inf),
 *             1 byte per element.
 *   MXC_E2M1: FP4 E2M1 elements (max 6), two per byte, the element at the
 *             even position in the low nibble.
 *   MXC_E2M3, MXC_E3M2: FP6 elements (OCP: E2M3 bias 1, max 7.5; E3M2 bias 3,
 *             max 28; no inf or NaN), packed as one little-endian bit string:
 *             the element at position p occupies bits 6p .. 6p+5 (bit 0 =
 *             least significant bit of byte 0), so 32 samples take 24 bytes.
 *             MicroQonv+ (Sec. IV-D, Tables II and VI) keeps activations
 *             in E3M2 with FP4 weights and gradients; the "-6" methods
 *             (Sec. VI-B, Tables VII and VIII) use E2M3 throughout.
 *             FP6 code buffers end with 16 bytes of slack that the library
 *             may read but never writes (included in mxconv_codes_bytes).
 *   Scales: one E8M0 byte per block, value 2^(code-127); 0xFF marks a block
 *   that held a NaN or infinity.
 *
 * Operand formats of the GEMM entry points (fwd, dgrad, wgrad and the fused
 * forms): `fmt` is either one format for both MX operands, or
 * MXC_PAIR(first, second) naming the format of each, in the order the call
 * takes them (fwd: W, X; dgrad: W, G_Y; wgrad: G_Y, X).  Supported: E4M3,
 * E2M1 and E2M3 alone, and MXC_PAIR(MXC_E2M1, MXC_E3M2) (MicroQonv+: FP4
 * weights or gradients against E3M2 activations); anything else returns
 * MXC_ERR_ARG.  (E3M2 against E3M2 is left out: the matrix cores do not sum
 * those products exactly.)  The FP6 forms run on the batch-block-32 kernels
 * (n a multiple of 32; fwd and dgrad: kernel width 1 or 3, fwd column
 * stride 1 or 2, dgrad stride 1x1 or 2x2); other layers return
 * MXC_ERR_SHAPE.
 *
 * Quantization rule (per block, the OCP-MX reading of Sec. III-A Eqs. (4)-(6)):
 *   s = clamp(floor(log2 max|x|) - emax, -127, 127), emax = 8 (E4M3), 2
 *   (E2M1, E2M3) or 4 (E3M2); scale code = s + 127 (code 0 when the block
 *   is all zero);
 *   element = x * 2^-s rounded to nearest, ties to even, saturating to the
 *   largest finite element; the sign of zero is kept; a non-finite block
 *   gets scale 0xFF and all-zero element codes.
 *
 * MX tensor layout ("MX-CBF").  A logical tensor (n, c, h, w) -- for weights
 * (Cout, Cin, Kh, Kw) -- is stored as
 *   codes  [Np/Bn][h][w][Cp][Bn]   (Bn fastest)
 *   scales [Np/Bn][h][w][Cp/32]
 * with Cp = c rounded up to 32.  One block = 32 channels x Bn batch samples at
 * one pixel (Sec. IV-A's X_{Cin,N}: at each (h, w) all channels of all
 * samples are contiguous; Sec. IV-B's square blocks along Cin and N).
 *   role MXC_ACT:    Bn = 32 if n >= 32 (n must be a multiple of 32),
 *                    else Bn = n (n must divide 32); Np = n.
 *                    E2M1 needs Bn >= 2, E2M3 and E3M2 Bn >= 4.
 *   role MXC_WEIGHT: Bn = 32, Np = n rounded up to 32, i.e. a block is
 *                    32 Cin x 32 Cout at one tap (Sec. IV-B: W_f is blocked
 *                    along Cin and Cout).
 * Padding channels / output channels hold +0 codes and never change a scale.
 *
 * Float layouts (mxc_layout) for quantize inputs and fwd/dgrad outputs:
 *   MXC_NCHW  plain (n, c, h, w) row-major (weights: OIHW);
 *   MXC_NHWC  (n, h, w, c);
 *   MXC_CBF   channel-batch-first fp32: [n/Bn][h][w][c][Bn] with the real c
 *             and the activation Bn above (Sec. IV-A's layout, unquantized).
 *   MXC_CBF_BF16  the same index order with bf16 elements: an output layout
 *             of mxconv_fwd, mxconv_dgrad and mxconv_backward for callers
 *             that keep their full-precision tensors in bf16.  The fp32
 *             GEMM result is rounded to the nearest bf16, ties to even (a
 *             NaN stays a NaN).  The quantize entry points read bf16 through
 *             their dtype argument and refuse this value (ARG).
 *
 * Convolution (mxc_conv): cross-correlation with zero padding, dilation 1,
 * groups 1; Ho = (h + 2 ph - kh) / sh + 1, Wo likewise (Sec. II-A, Eq. (1)
 * with the stride/padding the paper states the method is independent of).
 *
 * ---------------------------------------------------------------------------
 * Conventions for every entry point
 *   - Device pointers are caller-owned (allocated by the caller, e.g. as
 *     PyTorch tensors); the library never allocates, frees or synchronizes
 *     and keeps no state between calls beyond, per device, whether a kernel's
 *     large-LDS launch attribute has been raised (set once, safe to race).
 *     Calls from several host threads are safe.  All pointers to device
 *     memory must be 16-byte aligned.
 *   - Work is enqueued on `stream` (a hipStream_t passed as void*; NULL is
 *     the default stream) and runs asynchronously.
 *   - Arguments are validated on the host before anything is launched; a
 *     non-zero return means nothing was enqueued (except MXC_ERR_HIP).
 *   - Outputs are overwritten, never accumulated into.
 * Return codes: */
#ifndef MXCONV_H
#define MXCONV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MXC_OK             0
#define MXC_ERR_NULL      (-1)  /* a required pointer is NULL */
#define MXC_ERR_ARG       (-2)  /* bad enum value or non-positive size */
#define MXC_ERR_SHAPE     (-3)  /* batch rule broken, empty output, unsupported geometry */
#define MXC_ERR_ALIGN     (-4)  /* device pointer not 16-byte aligned */
#define MXC_ERR_HIP       (-5)  /* the HIP runtime reported a launch error */
#define MXC_ERR_WORKSPACE (-6)  /* workspace missing or smaller than required */

typedef enum { MXC_E4M3 = 0, MXC_E2M1 = 1, MXC_E2M3 = 2, MXC_E3M2 = 3 } mxc_fmt;
/* Different formats for the two MX operands of a GEMM entry point. */
#define MXC_PAIR(first, second) (0x10 | ((first) << 2) | (second))
typedef enum { MXC_F32 = 0, MXC_BF16 = 1 } mxc_dtype;
typedef enum { MXC_NCHW = 0, MXC_NHWC = 1, MXC_CBF = 2, MXC_CBF_BF16 = 3 } mxc_layout;
typedef enum { MXC_ACT = 0, MXC_WEIGHT = 1 } mxc_role;
typedef enum { MXC_FN_NONE = 0, MXC_FN_RELU = 1, MXC_FN_SILU = 2 } mxc_fn;   /* activation function */
/* Flag or-ed into mxconv_fwd_quant's fn: its fp32 output receives the values
 * before the activation (the pre-activation a backward pass needs for fn'). */
#define MXC_FN_PRE_OUT 0x100
/* Flag or-ed into the fn of mxconv_fwd_quant, mxconv_dgrad_quant and
 * mxconv_quantize_sum: the caller's full-precision tensors between layers
 * (pre-activations and input gradients) are bf16 CBF, and a GEMM result is
 * rounded to bf16 (as MXC_CBF_BF16) before anything uses it -- the value a
 * bf16 tensor would hold is the value that is activated, multiplied and
 * quantized.  Details with each entry point. */
#define MXC_FN_BF16 0x200

/* One convolution layer: batch n, channels cin -> cout, input h x w,
 * kernel kh x kw, stride sh, sw, zero padding ph, pw. */
typedef struct mxc_conv {
    int32_t n, cin, cout, h, w;
    int32_t kh, kw, sh, sw, ph, pw;
} mxc_conv;

/* ------------------------------------------------------------------ sizes */
/* Bytes of the code / scale arrays of an MX tensor (see layout above);
 * 0 if the arguments are invalid. */
size_t mxconv_codes_bytes(int role, int fmt, int n, int c, int h, int w);
size_t mxconv_scales_bytes(int role, int fmt, int n, int c, int h, int w);

/* Output spatial size of a layer; returns an error code. */
int mxconv_out_size(const mxc_conv* cv, int* ho, int* wo);

/* Bytes of the explicit CBF im2col codes / scales (mxconv_im2col_cbf). */
size_t mxconv_im2col_codes_bytes(const mxc_conv* cv, int fmt);
size_t mxconv_im2col_scales_bytes(const mxc_conv* cv, int fmt);

/* Workspace bytes mxconv_wgrad needs for its split-K partial sums (may be 0). */
size_t mxconv_wgrad_workspace_bytes(const mxc_conv* cv, int fmt);

/* ------------------------------------------------------------------ a1 */
/* Quantize a float tensor once into an MX tensor (Sec. III-A Eqs. (4)-(6) in
 * OCP-MX form, with Sec. IV-B's square blocks; Sec. IV-C: every tensor is
 * quantized once, activations before im2col).
 *   src     device, logical (n, c, h, w) tensor of `dtype` (fp32 or bf16) in
 *           `layout` (NCHW / NHWC / CBF; CBF only for role MXC_ACT).
 *           Weights are passed as OIHW (layout NCHW) with n = Cout, c = Cin,
 *           h = Kh, w = Kw.
 *   role    MXC_ACT (X, G_Y) or MXC_WEIGHT (W).
 *   codes   device, mxconv_codes_bytes(role, fmt, n, c, h, w) bytes, written.
 *   scales  device, mxconv_scales_bytes(...) bytes, written.
 * Errors: NULL, ARG (enum, sizes), SHAPE (batch rule), ALIGN, HIP. */
int mxconv_quantize(const void* src, int dtype, int layout, int role, int fmt,
                    int n, int c, int h, int w,
                    void* codes, uint8_t* scales, void* stream);

/* Flag for mxconv_quantize's `layout` (MXC_NCHW | MXC_KEEP_PAD): the codes of
 * the padding channels (c .. Cp - 1, which hold +0 codes) are not written.
 * The caller guarantees that `codes` already holds +0 codes there: a
 * zero-filled buffer, or one this call has filled before with the same
 * geometry.  For an input image (a few channels in one 32-channel block)
 * those rows are most of the stored codes: with c = 3, 29 of every 32 rows.
 * Only the few-channel NCHW path (role MXC_ACT, c <= 4, batch block 32,
 * FP8 or FP4) skips them; every other call writes them as usual, so the
 * result is the same either way. */
#define MXC_KEEP_PAD 0x100

/* Several quantizations in one call, with mxconv_quantize's rule: a layer's
 * forward operands (X and W), which become available together, are
 * quantized once each (Sec. IV-C) in a single launch.  Every job is exactly
 * an mxconv_quantize call (same arguments, same codes and scales); the jobs
 * that read a channel-batch-first activation with batch block 32 or OIHW
 * weights share one launch, any other job gets a launch of its own.  The
 * jobs' outputs must not overlap.
 *
 * A job may also ask for the channel-batch-first im2col of its activation
 * (a2): with `conv` non-NULL, `col_codes` / `col_scales` receive exactly
 * what mxconv_im2col_cbf(conv, fmt, codes, scales, ...) would write (layout
 * and sizes there).  For FP8 / FP4 activations read from the CBF layout with
 * batch block 32, the quantizer writes each block to its im2col positions as
 * it produces it (one launch for quantize and im2col, the codes not read
 * back); the wave of the block at pixel (y, x) also writes the zero blocks
 * of the padding taps of output pixel (y, x), which needs Ho <= h and
 * Wo <= w.  Any other such job is quantized and then copied by the im2col
 * kernel (a launch of its own after the quantizations).
 *   count  0 .. MXC_QMULTI_MAX;  jobs  host array of count descriptors.
 *   conv   NULL, or the layer whose input this job's tensor is: role
 *          MXC_ACT and (n, cin, h, w) equal to the job's (n, c, h, w).
 * Errors: as mxconv_quantize (checked for every job before anything is
 * launched), ARG for a count out of range, SHAPE for a conv that does not
 * match its job. */
#define MXC_QMULTI_MAX 24
typedef struct mxc_qjob {
    const void* src;
    int dtype, layout, role, fmt, n, c, h, w;
    void* codes;
    uint8_t* scales;
    const mxc_conv* conv;         /* optional im2col of the activation (NULL: none) */
    void* col_codes;
    uint8_t* col_scales;
} mxc_qjob;
int mxconv_quantize_multi(int count, const mxc_qjob* jobs, void* stream);

/* Quantize with stochastic rounding of the elements (Eq. (6) allows
 * round-to-nearest or stochastic rounding; Sec. III-A rounds gradients
 * stochastically and activations and weights to nearest).  Same arguments,
 * layout and scales as mxconv_quantize; each element becomes the upper of
 * its two neighbouring grid values lo <= |x| 2^-s < hi when r < frac * 2^16,
 * frac = (|x| 2^-s - lo) / (hi - lo), else the lower (sign kept; grid values
 * are exact; magnitudes at or above the format maximum saturate).  r: the 16
 * random bits of the code's linear position p in the code array: Philox4x32-10
 * (Salmon et al., SC'11) with key (seed mod 2^32, seed / 2^32) and counter
 * (p / 8 mod 2^32, p / 2^35, 0, 0) gives words w0..w3, and j = p mod 8 takes
 * bits 16 (j mod 2) .. 16 (j mod 2) + 15 of w[j / 2].  The same seed and
 * tensor always give the same codes, whatever the source layout.
 * Errors: as mxconv_quantize. */
int mxconv_quantize_sr(const void* src, int dtype, int layout, int role, int fmt,
                       int n, int c, int h, int w, uint64_t seed,
                       void* codes, uint8_t* scales, void* stream);

/* ------------------------------------------------------------------ f4 */
/* The paper's own two-level NVFP format, Eqs. (4)-(6) literally (Sec.
 * III-A, with Sec. IV-B's square blocks of B = 64 = 8 x 8):
 *   T = amax / (448 * emax_val)            per tensor (Eq. (4)), fp32;
 *   B = CastE4M3(bmax / (T * emax_val))    per 8-channel x 8-sample block
 *                                          (weights: 8 Cin x 8 Cout at one
 *                                          tap), E4M3 to nearest even,
 *                                          saturating at 448 (Eq. (5));
 *   code = Round(x / (B * T))              to nearest even, saturating
 *                                          (Eq. (6));
 * each step one IEEE fp32 operation (divisions correctly rounded), emax_val
 * the element format's largest value (448, 6, 7.5 or 28).  T = 0 or B = 0
 * gives zero codes; a non-finite element makes T NaN, every block scale
 * 0x7F and every code 0.  Dequantized value: code value x B x T.
 *   codes    device, mxconv_codes_bytes(role, fmt, ...) bytes, the MX-CBF
 *            code layout.
 *   scales   device, mxconv_nvfp_scales_bytes(...) E4M3 bytes in the layout
 *            [Np/Bn][h][w][Cp/8][Bn/8].
 *   tscale   device, one float: T.
 *   workspace device, >= mxconv_nvfp_workspace_bytes() bytes, scratch.
 * The GPU kernels take CBF activations with batch block 32 or OIHW weights
 * (layout MXC_NCHW, role MXC_WEIGHT); other sources return MXC_ERR_SHAPE.
 * Two launches on `stream` (per-workgroup maxima, then the quantization).
 * Errors: NULL, ARG, SHAPE, WORKSPACE, ALIGN, HIP. */
size_t mxconv_nvfp_scales_bytes(int role, int fmt, int n, int c, int h, int w);
size_t mxconv_nvfp_workspace_bytes(void);
int mxconv_nvfp_quantize(const void* src, int dtype, int layout, int role, int fmt,
                         int n, int c, int h, int w, void* codes, uint8_t* scales,
                         float* tscale, void* workspace, size_t ws_bytes, void* stream);

/* The three GEMMs on NVFP operands (element codes with E4M3 8x8 block
 * scales and per-tensor scales, as mxconv_nvfp_quantize writes them): Y =
 * W * X, G_X = W^T * G_Y, G_W = G_Y * X^T (Eqs. (1)-(3)) of the
 * fake-quantized tensors code x B x T.  The block-scaled matrix cores take
 * only E8M0 scales per 32 elements, so the kernels decode each fragment --
 * to fp16 for FP4 and FP6 elements, to bf16 for FP8 (code x B is exact in
 * either) -- run fp16 / bf16 MFMAs with fp32 accumulation and multiply the
 * result by the two per-tensor scales.  Arguments as mxconv_fwd / dgrad /
 * wgrad, with each operand's E4M3 block scales (mxconv_nvfp_scales_bytes)
 * and its per-tensor scale (w_t, x_t, gy_t: device floats).  fmt: one
 * format for both operands -- MXC_E2M1 (NVFP4, the paper's format),
 * MXC_E2M3 (NVFP6 of the "-6" methods, Sec. VI-B), MXC_E4M3 (NVFP8) -- or
 * MXC_PAIR(MXC_E2M1, MXC_E3M2), FP4 weights or gradients with E3M2
 * activations (MicroQonv+, Sec. IV-D), in the operand order of the call
 * (W, X / W, G_Y / G_Y, X); other pairs return MXC_ERR_ARG.  Layers outside
 * the batch-block-32 kernels (kernel width 1 or 3, forward column stride 1
 * or 2, input-gradient stride 1x1 or 2x2) return MXC_ERR_SHAPE.  The weight
 * gradient uses the workspace of mxconv_wgrad_workspace_bytes(cv, fmt).
 * Errors: NULL, ARG, SHAPE, ALIGN, WORKSPACE, HIP. */
int mxconv_nvfp_fwd(const mxc_conv* cv, int fmt,
                    const void* w_codes, const uint8_t* w_scales, const float* w_t,
                    const void* x_codes, const uint8_t* x_scales, const float* x_t,
                    float* y, int y_layout, void* stream);
int mxconv_nvfp_dgrad(const mxc_conv* cv, int fmt,
                      const void* w_codes, const uint8_t* w_scales, const float* w_t,
                      const void* gy_codes, const uint8_t* gy_scales, const float* gy_t,
                      float* gx, int gx_layout, void* stream);
int mxconv_nvfp_wgrad(const mxc_conv* cv, int fmt,
                      const void* gy_codes, const uint8_t* gy_scales, const float* gy_t,
                      const void* x_codes, const uint8_t* x_scales, const float* x_t,
                      float* gw, void* workspace, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------ a2 */
/* Channel-batch-first im2col on MX codes (Sec. IV-A, X'_{Cin,N}): for every
 * output pixel (ho, wo) and tap (kh, kw), the block of the input pixel
 * (ho*sh+kh-ph, wo*sw+kw-pw) is copied whole -- codes and scale, no
 * requantization; taps in the zero padding give all-zero blocks with scale
 * code 0.
 *   x_codes / x_scales   device, the quantized activation (role ACT,
 *                        n = cv->n, c = cv->cin, h = cv->h, w = cv->w).
 *   col_codes            device, [n/Bn][Ho][Wo][Kh][Kw][Cp][Bn] codes,
 *                        mxconv_im2col_codes_bytes bytes.
 *   col_scales           device, [n/Bn][Ho][Wo][Kh][Kw][Cp/32],
 *                        mxconv_im2col_scales_bytes bytes.
 * Errors: NULL, ARG, SHAPE, ALIGN, HIP. */
int mxconv_im2col_cbf(const mxc_conv* cv, int fmt,
                      const void* x_codes, const uint8_t* x_scales,
                      void* col_codes, uint8_t* col_scales, void* stream);

/* ------------------------------------------------------------------ a3 */
/* Forward convolution Y = W * X (Eq. (1)) as the GEMM Y_f = W_f X'
 * (Sec. II-C, with Sec. IV-B's reshaping), the im2col being implicit: the
 * kernel reads the X blocks of each tap straight from the MX-CBF tensor.
 * Each 32-element K block is multiplied with its two E8M0 scales as in
 * Eq. (7); accumulation is fp32.
 *   w_codes / w_scales   device, W quantized with role MXC_WEIGHT
 *                        (n = cout, c = cin, h = kh, w = kw).
 *   x_codes / x_scales   device, X quantized with role MXC_ACT.
 *   y                    device, n x cout x Ho x Wo in y_layout
 *                        (fp32 MXC_NCHW or MXC_CBF, or bf16 MXC_CBF_BF16).
 * Errors: NULL, ARG, SHAPE, ALIGN, HIP. */
int mxconv_fwd(const mxc_conv* cv, int fmt,
               const void* w_codes, const uint8_t* w_scales,
               const void* x_codes, const uint8_t* x_scales,
               void* y, int y_layout, void* stream);

/* ------------------------------------------------------------------ a4 */
/* Input gradient G_X = W^T * G_Y (Eq. (2)), i.e. G_X' = W_f^T G_Yf followed
 * by the col2im that folds G_X' back onto input pixels (Sec. II-C,
 * Sec. IV-B).  Computed as an implicit transposed convolution: for each
 * input pixel the kernel gathers the G_Y blocks of the taps that reach it,
 * so nothing is scattered.  Operands are the same stored codes as in the
 * forward pass (W) and the once-quantized G_Y.
 *   gy_codes / gy_scales  device, G_Y quantized with role MXC_ACT
 *                         (n, cout, Ho, Wo).
 *   gx                    device, n x cin x h x w in gx_layout
 *                         (fp32 MXC_NCHW or MXC_CBF, or bf16 MXC_CBF_BF16).
 * Errors: NULL, ARG, SHAPE, ALIGN, HIP. */
int mxconv_dgrad(const mxc_conv* cv, int fmt,
                 const void* w_codes, const uint8_t* w_scales,
                 const void* gy_codes, const uint8_t* gy_scales,
                 void* gx, int gx_layout, void* stream);

/* ------------------------------------------------------------------ a5 */
/* Weight gradient G_W[co][ci] = sum_n G_Y[n][co] * X[n][ci] (Eq. (3)), i.e.
 * G_Wf = G_Yf X'^T (Sec. II-C, Sec. IV-B), contracted over (pixel, sample)
 * with one 32-element K block per pixel's batch block, reading the same
 * once-quantized X codes as the forward pass.  Split over K across the GPU;
 * partial sums go to `workspace` and are reduced in fp32.
 *   gw          device fp32, cout x cin x kh x kw (OIHW), written.
 *   workspace   device, >= mxconv_wgrad_workspace_bytes(cv, fmt) bytes
 *               (may be NULL when that is 0); contents are scratch.
 * Errors: NULL, ARG, SHAPE, ALIGN, WORKSPACE, HIP. */
int mxconv_wgrad(const mxc_conv* cv, int fmt,
                 const void* gy_codes, const uint8_t* gy_scales,
                 const void* x_codes, const uint8_t* x_scales,
                 float* gw, void* workspace, size_t ws_bytes, void* stream);

/* The weight gradient in two parts, for callers that finish several layers'
 * weight gradients together (at the end of a backward pass, say):
 * mxconv_wgrad_deferred takes mxconv_wgrad's arguments and runs its GEMM but
 * leaves the split-K partial sums in the workspace (a layer without split
 * gets its G_W written directly); mxconv_wgrad_reduce_multi then finishes up
 * to MXC_WREDUCE_MAX such layers with one launch.  The result is bit for bit
 * mxconv_wgrad's (the same partial sums, added in the same order).  Each job
 * names the layer and format of its deferred call, that call's workspace
 * (untouched in between) and G_W; the reduction must follow the deferred
 * calls on the stream.
 * Errors: as mxconv_wgrad for every job (checked before anything is
 * launched), ARG for a count out of range. */
#define MXC_WREDUCE_MAX 32
typedef struct mxc_wjob {
    const mxc_conv* conv;
    int fmt;
    const void* workspace;
    size_t ws_bytes;
    float* gw;
} mxc_wjob;
int mxconv_wgrad_deferred(const mxc_conv* cv, int fmt,
                          const void* gy_codes, const uint8_t* gy_scales,
                          const void* x_codes, const uint8_t* x_scales,
                          float* gw, void* workspace, size_t ws_bytes, void* stream);
int mxconv_wgrad_reduce_multi(int count, const mxc_wjob* jobs, void* stream);

/* Both gradients of one layer (Eqs. (2) and (3), Sec. II-C) from one call:
 * mxconv_dgrad's result in gx and mxconv_wgrad's (deferred = 0) or
 * mxconv_wgrad_deferred's (deferred = 1) in gw / workspace, bit for bit.
 * Both products read the same quantized G_Y; with batch block 32, kernel
 * width 1 or 3, stride 1 or 2 and format MXFP8 or MXFP4 they run as one
 * launch, otherwise as the two calls one after the other.
 *   fmt              passed to both products as their fmt (so the pair
 *                    (W, G_Y) and the pair (G_Y, X) have the same formats).
 *                    A mixed MXC_PAIR(a, b) with a != b is refused (ARG):
 *                    G_Y would have to be read as b by the input gradient
 *                    and as a by the weight gradient.
 *   w_*, gy_*, x_*   as for mxconv_dgrad and mxconv_wgrad; gx, gx_layout as
 *                    for mxconv_dgrad; gw, workspace, ws_bytes as for
 *                    mxconv_wgrad.
 * Errors: NULL, ARG (also deferred not 0 or 1), SHAPE, WORKSPACE, ALIGN, HIP,
 * all checked before anything is launched. */
int mxconv_backward(const mxc_conv* cv, int fmt,
                    const void* w_codes, const uint8_t* w_scales,
                    const void* gy_codes, const uint8_t* gy_scales,
                    const void* x_codes, const uint8_t* x_scales,
                    void* gx, int gx_layout, float* gw,
                    void* workspace, size_t ws_bytes, int deferred, void* stream);

/* ------------------------------------------------------------------ a6 */
/* Naive comparator (the baseline of Sec. III-C and Table I): the im2col is
 * done in full precision first, and every GEMM operand is then quantized
 * with 1-D blocks of 32 elements along that GEMM's contraction dimension --
 * so X', W and G_Y are each quantized twice per step, once per GEMM they
 * enter.  Same element formats and scale rule as above; only the block shape
 * and the data flow differ.  It exists to be measured against, not used.
 *
 * Matrices are in channels-last GEMM form: P = n*Ho*Wo output positions
 * ordered (n, ho, wo); K = kh*kw*cin ordered (kh, kw, ci).  X, G_Y and G_X
 * are NHWC fp32 (G_Y is then [P][cout]); W and G_W are OHWI fp32, i.e.
 * [cout][K].
 *
 * Line matrix: the output of mxconv_naive_quantize_1d.  A matrix blocked
 * along one dimension of length L is stored with that dimension contiguous:
 *   codes  [lines][Lp]     (FP4: two per byte, even element in the low nibble)
 *   scales [lines][Lp/32]
 * Lp = L rounded up to a multiple of 64 (padding codes and scales are 0). */

/* Bytes of a line matrix of `lines` lines of length `len`; 0 if invalid. */
size_t mxconv_naive_codes_bytes(int64_t lines, int64_t len, int fmt);
size_t mxconv_naive_scales_bytes(int64_t lines, int64_t len);

/* fp32 im2col: col[p][k] = x[n][ho*sh+kh-ph][wo*sw+kw-pw][ci], 0 in the
 * padding (Eq. (1) unrolled into the GEMM of Sec. II-C).
 *   x    device fp32, NHWC (n, h, w, cin).
 *   col  device fp32, [P][K], written.
 * Errors: NULL, ARG, SHAPE, ALIGN, HIP. */
int mxconv_naive_im2col_f32(const mxc_conv* cv, const float* x, float* col, void* stream);

/* 1-D quantization of a row-major fp32 matrix src[rows][cols].
 *   dir 0: blocks of 32 along each row    -> lines = rows, L = cols;
 *   dir 1: blocks of 32 down each column  -> lines = cols, L = rows (the
 *          output is the transposed line matrix).
 *   codes   device, mxconv_naive_codes_bytes(lines, L, fmt) bytes, written.
 *   scales  device, mxconv_naive_scales_bytes(lines, L) bytes, written.
 * Errors: NULL, ARG, ALIGN, HIP. */
int mxconv_naive_quantize_1d(const float* src, int64_t rows, int64_t cols, int dir, int fmt,
                             void* codes, uint8_t* scales, void* stream);

/* Forward GEMM Y[P][cout] = X'[P][K] W[cout][K]^T (Sec. II-C), both operands
 * blocked along K:
 *   col_codes / col_scales  X' quantized with dir 0 (lines P, length K);
 *   w_codes / w_scales      W (OHWI as [cout][K]) quantized with dir 0;
 *   y                       device fp32 [P][cout] (= NHWC), written.
 * Errors: NULL, ARG, SHAPE, ALIGN, HIP. */
int mxconv_naive_fwd(const mxc_conv* cv, int fmt,
                     const void* col_codes, const uint8_t* col_scales,
                     const void* w_codes, const uint8_t* w_scales,
                     float* y, void* stream);

/* Input gradient: G_X'[P][K] = G_Y[P][cout] W[cout][K] (Sec. II-C), both
 * blocked along cout, then col2im (sum over the taps that read each input
 * element):
 *   gy_codes / gy_scales  G_Y ([P][cout]) quantized with dir 0;
 *   wt_codes / wt_scales  W ([cout][K]) quantized with dir 1 (lines K);
 *   gcol                  device fp32 [P][K] scratch for G_X';
 *   gx                    device fp32 NHWC (n, h, w, cin), written.
 * Errors: NULL, ARG, SHAPE, ALIGN, HIP. */
int mxconv_naive_dgrad(const mxc_conv* cv, int fmt,
                       const void* gy_codes, const uint8_t* gy_scales,
                       const void* wt_codes, const uint8_t* wt_scales,
                       float* gcol, float* gx, void* stream);

/* Weight gradient: G_W[cout][K] = G_Y[P][cout]^T X'[P][K] (Sec. II-C), both
 * blocked along P:
 *   gyt_codes / gyt_scales  G_Y ([P][cout]) quantized with dir 1 (lines cout);
 *   xt_codes / xt_scales    X' ([P][K]) quantized with dir 1 (lines K);
 *   gw                      device fp32 [cout][K] (= OHWI), written.
 * Errors: NULL, ARG, SHAPE, ALIGN, HIP. */
int mxconv_naive_wgrad(const mxc_conv* cv, int fmt,
                       const void* gyt_codes, const uint8_t* gyt_scales,
                       const void* xt_codes, const uint8_t* xt_scales,
                       float* gw, void* stream);

/* ------------------------------------------------------------------ f1 */
/* Fused quantizing epilogues.  In the paper's training step a layer's output
 * is still on chip when it is quantized for the next use, and only the MX
 * codes go off chip (Sec. V, DRAM simulation; Sec. IV-B: every tensor is
 * quantized once).  Here the forward and input-gradient kernels quantize
 * their output tile in the epilogue: one 32-channel x 32-sample output tile
 * at one pixel is exactly one MX block of the next consumer's operand, so
 * the block maximum, E8M0 scale and codes are formed in registers with the
 * rule of mxconv_quantize (role MXC_ACT) and no fp32 tensor is written.
 *
 * Forward: Y = fn(W * X), fn in mxc_fn (MXC_FN_NONE, MXC_FN_RELU, or
 * MXC_FN_SILU y / (1 + exp(-y))), quantized into the MX-CBF tensor of
 * (n, cout, Ho, Wo):
 *   y_codes / y_scales  device, mxconv_codes_bytes / mxconv_scales_bytes(
 *                       MXC_ACT, out_fmt, n, cout, Ho, Wo) bytes, written
 *                       (out_fmt any mxc_fmt; FP6 slack not written).
 *   y_act               NULL, or device fp32 n x cout x Ho x Wo in CBF
 *                       layout: receives the values that were quantized,
 *                       or, with fn | MXC_FN_PRE_OUT, W * X before fn.
 *                       With fn | MXC_FN_BF16, W * X is rounded to bf16
 *                       first and fn applied to that; y_act with
 *                       MXC_FN_PRE_OUT is then bf16 CBF and receives the
 *                       rounded W * X (the pre-activation a bf16 network
 *                       keeps), without it fp32 as above.
 * Input gradient: G_Z = (W^T * G_Y) . fn'(z), the gradient at the
 * pre-activation z of this layer's input X = fn(z) (fn' = 1 for
 * MXC_FN_NONE, [z > 0] for ReLU, s (1 + z (1 - s)) with s = 1 / (1 +
 * exp(-z)) for SiLU), quantized into the MX-CBF tensor of (n, cin, h, w) --
 * the G_Y operand of the layer before:
 *   z                   device fp32 n x cin x h x w in CBF layout; may be
 *                       NULL for MXC_FN_NONE.  With fn | MXC_FN_BF16, z is
 *                       bf16 CBF and W^T * G_Y is rounded to bf16 before
 *                       the product (so the result equals mxconv_dgrad into
 *                       MXC_CBF_BF16 followed by mxconv_quantize_sum).
 *   gx_codes / gx_scales, gx_act  as above for (n, cin, h, w); gx_act is
 *                       fp32 in both modes.
 * The fused kernels cover batch block 32 (n a multiple of 32), kernel width
 * 1 or 3, forward column stride 1 or 2, input-gradient stride 1x1 or 2x2;
 * other layers return MXC_ERR_SHAPE (use mxconv_fwd / mxconv_dgrad and
 * mxconv_quantize).
 * Errors: NULL, ARG, SHAPE, ALIGN, HIP. */
int mxconv_fwd_quant(const mxc_conv* cv, int fmt,
                     const void* w_codes, const uint8_t* w_scales,
                     const void* x_codes, const uint8_t* x_scales,
                     int fn, int out_fmt, void* y_codes, uint8_t* y_scales,
                     void* y_act, void* stream);
int mxconv_dgrad_quant(const mxc_conv* cv, int fmt,
                       const void* w_codes, const uint8_t* w_scales,
                       const void* gy_codes, const uint8_t* gy_scales,
                       int fn, const void* z, int out_fmt,
                       void* gx_codes, uint8_t* gx_scales, float* gx_act, void* stream);
/* mxconv_dgrad_quant with the gradient's element codes rounded
 * stochastically (Sec. III-A rounds gradients stochastically; Eq. (6)):
 * the scales, the fp32 values (gx_act) and every other argument as
 * mxconv_dgrad_quant; each code is the rule of mxconv_quantize_sr applied to
 * the value gx_act receives, with the random bits of its linear position in
 * the gx_codes array under `seed` -- so the codes equal mxconv_quantize_sr of
 * gx_act (CBF, role MXC_ACT) with the same seed.
 * Errors: as mxconv_dgrad_quant. */
int mxconv_dgrad_quant_sr(const mxc_conv* cv, int fmt,
                          const void* w_codes, const uint8_t* w_scales,
                          const void* gy_codes, const uint8_t* gy_scales,
                          int fn, const void* z, int out_fmt,
                          void* gx_codes, uint8_t* gx_scales, float* gx_act, uint64_t seed, void* stream);

/* ------------------------------------------------------------------ no allocation */
/* mxconv_wgrad for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * Same arguments and results as mxconv_wgrad without the workspace: the
 * split-K partial sums go to a library-owned device array of
 * MXC_NOALLOC_WS_MAX bytes that every GPU the library runs on holds until
 * the process ends (its address on a device is looked up on the first call
 * made with that device current).  The call itself allocates nothing.
 * Calls that overlap in time on one GPU (different streams or host threads)
 * share that array and race; the array keeps the last call's partial sums.
 * Errors: as mxconv_wgrad; WORKSPACE when the layer needs more than
 * MXC_NOALLOC_WS_MAX bytes (mxconv_wgrad_workspace_bytes), checked before
 * any launch. */
#define MXC_NOALLOC_WS_MAX (16u << 20)
int mxconv_wgrad_noalloc(const mxc_conv* cv, int fmt,
                         const void* gy_codes, const uint8_t* gy_scales,
                         const void* x_codes, const uint8_t* x_scales,
                         float* gw, void* stream);

/* ------------------------------------------------------------------ network steps */
/* Between the convolutions of a whole network's training step (the YOLO
 * backbone + neck and the latent-replay stacks of Sec. VI-VII), two more
 * operations touch activations and gradients; both keep every tensor
 * quantized exactly once (Sec. IV-C).
 *
 * Channel concatenation and nearest-neighbour 2x upsampling of MX-CBF
 * activations.  A block is 32 channels x Bn samples at one pixel (Sec. IV-A,
 * IV-B), so both are index maps on whole blocks: codes and E8M0 scales are
 * copied, never requantized.  The destination is the MX-CBF tensor of
 * (n, 32 * sum_k ncb_k, h, w) (role MXC_ACT, format fmt): part k fills the
 * channel blocks [off_k, off_k + ncb_k), off_k = sum_{i<k} ncb_i, in order,
 * so a part whose channel count is not a multiple of 32 brings its zero
 * padding channels along as channels of the destination.
 *   part.codes/scales  device MX-CBF tensor (n, c_k, h_k, w_k) of format fmt
 *                      (the same batch block as the destination);
 *   part.ncb           ceil(c_k / 32);
 *   part.up            0: (h_k, w_k) = (h, w); 1: (h_k, w_k) = (h/2, w/2) and
 *                      destination pixel (y, x) reads source pixel
 *                      (y/2, x/2) (h and w even).
 *   codes / scales     device, written (mxconv_codes_bytes /
 *                      mxconv_scales_bytes of the destination).
 * 1 <= nparts <= MXC_CONCAT_MAX.  Errors: NULL, ARG, SHAPE, ALIGN, HIP. */
#define MXC_CONCAT_MAX 4
typedef struct {
    const void* codes;
    const uint8_t* scales;
    int ncb;
    int up;
} mxc_part;
int mxconv_concat_cbf(int fmt, int n, int h, int w, int nparts, const mxc_part* parts,
                      void* codes, uint8_t* scales, void* stream);

/* Quantize the gradient of a tensor a = fn(z) read by several consumers:
 *   G = fn'(z) . (t_0 + t_1 + ... + t_{nterms-1})
 * (fn' as for mxconv_dgrad_quant; z may be NULL for MXC_FN_NONE), quantized
 * once with the rule of mxconv_quantize (role MXC_ACT) into the MX-CBF tensor
 * of (n, c, h, w) -- the G_Y operand of the layer that produced a.  Each term
 * is read from an fp32 CBF tensor [n/32][hs][ws][c_src][32] -- a consumer's
 * input gradient:
 *   term.src     device fp32 (see MXC_FN_BF16 below);
 *   term.c_src   channels of that tensor; term.c_off: its channel that is
 *                channel 0 of the term (c_off + c <= c_src: the slice a
 *                concatenation's gradient hands back to one part);
 *   term.down    0: (hs, ws) = (h, w); 1: (hs, ws) = (2h, 2w) and the term
 *                at (y, x) is (s(2y,2x) + s(2y,2x+1)) + (s(2y+1,2x) +
 *                s(2y+1,2x+1)) -- the gradient of a 2x upsampling.
 * The fp32 sum runs over the terms in order (((t_0 + t_1) + t_2) + ...).
 *   z            device fp32 CBF [n/32][h][w][c][32], the pre-activation;
 *   codes/scales device, written;
 *   vals         NULL, or device fp32 CBF [n/32][h][w][c][32]: receives G.
 * With fn | MXC_FN_BF16 every term and z are bf16 CBF instead (read
 * exactly; the sum, the product and vals stay fp32).
 * n a multiple of 32; fmt MXC_E4M3 or MXC_E2M1; 1 <= nterms <= MXC_TERMS_MAX.
 * Errors: NULL, ARG, SHAPE, ALIGN, HIP. */
#define MXC_TERMS_MAX 4
typedef struct {
    const void* src;       /* fp32, or bf16 with MXC_FN_BF16 */
    int c_src;
    int c_off;
    int down;
} mxc_term;
int mxconv_quantize_sum(int fmt, int n, int c, int h, int w, int nterms, const mxc_term* terms,
                        int fn, const void* z, void* codes, uint8_t* scales, float* vals, void* stream);
/* mxconv_quantize_sum with stochastic rounding of the gradient's elements
 * (Sec. III-A; Eq. (6)): the same sum, product, scales and vals; each code is
 * the rule of mxconv_quantize_sr applied to the value vals receives, keyed by
 * its linear position in the code array under `seed` (so the codes equal
 * mxconv_quantize_sr of vals, CBF, role MXC_ACT, with the same seed).
 * Errors: as mxconv_quantize_sum. */
int mxconv_quantize_sum_sr(int fmt, int n, int c, int h, int w, int nterms, const mxc_term* terms,
                           int fn, const void* z, void* codes, uint8_t* scales, float* vals, uint64_t seed,
                           void* stream);

/* Human-readable text for a return code (static storage). */
const char* mxconv_strerror(int code);

#ifdef __cplusplus
}
#endif
#endif /* MXCONV_H */
