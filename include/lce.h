/*
 * lce.h - C ABI of the MI355X (gfx950) bitpacked binary 2-D convolution.
 *
 * The operator is LceBConv2d of Larq Compute Engine (arXiv 2011.09398,
 * Section 3.2, "Operator implementations"), preceded by the sign
 * binarization and bitpacking of LceQuantize (same section):
 *
 *   1. bitpack:   bit = 1 (standing for -1.0) iff x < 0, else 0 (+1.0);
 *                 channel c goes to 32-bit word c/32, bit c%32; the channel
 *                 count is padded up to a multiple of 32 with 0 bits.
 *   2. im2col over the bitpacked NHWC tensor, padded locations read as
 *      0 bits, i.e. +1.0 ("one-padding"), or, on request, as 0.0
 *      (TensorFlow's zero padding, through a correction step).
 *   3. XOR + POPCOUNT GEMM against bitpacked +-1 filters:
 *          dot = K - 2 * sum_k popcount(a_k XOR w_k),  K = KH*KW*C_in.
 *   4. fused output transform on the integer accumulator:
 *          c = min(max(dot, clamp_min), clamp_max)   (fused activation)
 *          float32 output:   y = fmaf((float)c, multiplier[co], bias[co])
 *          bitpacked output: bit = 1 iff c < thresholds[co] (exact compare),
 *                            optionally inverted per channel
 *
 * Conventions shared by every entry point:
 *   - All tensor pointers are DEVICE pointers owned by the caller.  The
 *     library never allocates, frees or synchronizes; all work is enqueued
 *     asynchronously on `stream` (NULL = the default stream).
 *   - Activations are NHWC, filters OHWI (the TensorFlow Lite orders), and a
 *     bitpacked tensor stores ceil(C/32) int32 words per pixel (or filter
 *     tap) with its packed-channel axis innermost.  Bits beyond the real
 *     channel count MUST be zero in every bitpacked input; lce_bitpack and
 *     lce_bconv2d's bitpacked output always write them as zero.
 *   - Outputs must not alias inputs.
 *   - Arguments are validated on the host before anything is launched; on
 *     any error nothing is written or launched, the status is returned, and
 *     lce_last_error() describes it.  Asynchronous device faults surface at
 *     the caller's next synchronization.  No C++ exception crosses the ABI.
 */
#ifndef LCE_H_
#define LCE_H_

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    LCE_OK = 0,
    LCE_EINVAL = 1,        /* null pointer, bad size or enum, empty output   */
    LCE_EUNSUPPORTED = 2,  /* well-formed request the library does not run   */
    LCE_EALIGN = 3,        /* pointer not aligned to its element type        */
    LCE_EHIP = 4           /* the HIP runtime reported an error at launch    */
} lce_status;

/* Spatial padding, TensorFlow semantics: SAME gives ceil(H/stride) outputs
 * with floor(total/2) padding before and the rest after; VALID none. */
typedef enum { LCE_PADDING_VALID = 0, LCE_PADDING_SAME = 1 } lce_padding;

/* Value read at padded locations.  ONE (0 bits, +1.0) is the one-padding of
 * Section 3.2, the fast path.  ZERO is TensorFlow's zero padding, which the
 * same section supports through a correction step: the padded taps are
 * computed as +1.0 and their filter sums are taken out again, using the
 * table of lce_bconv2d_pad_correction. */
typedef enum { LCE_PAD_ONE = 0, LCE_PAD_ZERO = 1 } lce_pad_value;

/* Output of lce_bconv2d:
 *   FLOAT32   float  [N][OH][OW][C_out]
 *   BITPACKED int32  [N][OH][OW][ceil(C_out/32)]
 *   INT32     int32  [N][OH][OW][C_out], the clamped accumulator c itself */
typedef enum { LCE_OUT_FLOAT32 = 0, LCE_OUT_BITPACKED = 1, LCE_OUT_INT32 = 2 } lce_out_type;

/* One binary convolution.  Every field is a plain int32 (enums by value). */
typedef struct {
    int32_t n, h, w, c_in;          /* input activations, NHWC, >= 1          */
    int32_t c_out, kh, kw;          /* filters, OHWI, >= 1                    */
    int32_t stride_h, stride_w;     /* >= 1                                   */
    int32_t padding;                /* lce_padding                            */
    int32_t pad_value;              /* lce_pad_value                          */
    int32_t clamp_min, clamp_max;   /* fused activation bounds on the integer
                                       accumulator; clamp_min <= clamp_max.
                                       INT32_MIN/INT32_MAX = no activation    */
    int32_t out_type;               /* lce_out_type                           */
} lce_bconv2d_desc;

/* Number of 32-bit words holding `channels` packed channels: ceil(c/32)
 * (Section 3.2, LceQuantize: the channel count is padded up to a multiple of
 * 32 and every 32 channels become one word).  Returns -1 when channels < 0. */
int32_t lce_packed_words(int32_t channels);

/* Output height/width of `desc`.  LceBConv2d extends TensorFlow Lite's
 * convolution (Section 3, Section 3.2), so its geometry is TensorFlow's:
 * SAME gives ceil(H/stride) rows, VALID floor((H-KH)/stride)+1, and likewise
 * for the width.  Validates the descriptor exactly as lce_bconv2d does,
 * except for pointers.
 * Errors: LCE_EINVAL (null desc/oh/ow, bad field, no output). */
lce_status lce_bconv2d_out_shape(const lce_bconv2d_desc *desc, int32_t *oh, int32_t *ow);

/* LceQuantize (Section 3.2): sign-binarize and bitpack a row-major float
 * array x[rows][channels] into out[rows][ceil(channels/32)].
 * Bit c%32 of word c/32 is 1 iff x[r][c] < 0.0f (so -0.0 and NaN give 0,
 * i.e. +1.0); the bits past `channels` are written as 0.
 * For activations rows = N*H*W; for OHWI filters (the 1-bit weight storage
 * of Section 3.1) rows = C_out*KH*KW with channels = C_in.
 * rows == 0 is a no-op (pointers may then be NULL).  x must be 4-byte
 * aligned (16-byte alignment and a channel count that is a multiple of 32
 * take the fastest path), out 4-byte.
 * Errors: LCE_EINVAL (null pointer, rows < 0, channels < 1),
 *         LCE_EALIGN, LCE_EHIP. */
lce_status lce_bitpack(const float *x, int32_t *out, int64_t rows, int32_t channels,
                       hipStream_t stream);

/* LceBConv2d (Section 3.2): bitpacked binary convolution with the fused
 * output transform.
 *   x_packed   int32 [N][H][W][ceil(C_in/32)]          (device)
 *   w_packed   int32 [C_out][KH][KW][ceil(C_in/32)]    (device)
 *   multiplier float [C_out] or NULL (= 1.0)   used by FLOAT32 output only
 *   bias       float [C_out] or NULL (= 0.0)   used by FLOAT32 output only
 *   thresholds float [C_out], required by BITPACKED output only
 *   flip       int32 [ceil(C_out/32)] or NULL, used by BITPACKED output
 *              only: output bits of the channels whose bit is set here are
 *              inverted (bit = NOT(c < thresholds[co])), the direction that
 *              lce_fold_thresholds derives from a negative multiplier.  Bits
 *              past C_out are ignored.
 *   pad_correction int32 table from lce_bconv2d_pad_correction for these
 *              filters; required when pad_value is ZERO and some window
 *              reaches outside the image (SAME with a nonzero total padding),
 *              ignored (may be NULL) otherwise
 *   out        see lce_out_type; shape from lce_bconv2d_out_shape
 * Dilation and groups are not part of the operator (always 1).
 * All pointers must be 4-byte aligned.
 * Errors: LCE_EINVAL (null desc or required pointer, bad field, no output,
 *         c_out > 2^20, a tensor of 2^31 or more words/elements; with zero
 *         padding also K >= 2^29), LCE_EALIGN, LCE_EHIP. */
lce_status lce_bconv2d(const lce_bconv2d_desc *desc,
                       const int32_t *x_packed, const int32_t *w_packed,
                       const float *multiplier, const float *bias,
                       const float *thresholds, const int32_t *flip,
                       const int32_t *pad_correction, void *out, hipStream_t stream);

/* LceQuantize followed by the LceBConv2d that consumes it, in one launch
 * (Section 3.2: the float activation is sign-binarized and bitpacked, then
 * convolved).  The result equals lce_bitpack of x followed by lce_bconv2d
 * on the packed tensor, bit for bit, with no packed copy written to memory:
 * each workgroup binarizes the input rows its own windows read.  That work
 * is repeated by every filter group, so this pays at small batches, where
 * a separate lce_bitpack launch costs more than it.
 *   x          float32 [N][H][W][C_in]  (device, 16-byte aligned); the sign
 *              test is lce_bitpack's (x < 0.0f is a 1 bit = -1.0, so -0.0
 *              and NaN give +1.0)
 *   w_packed, multiplier, bias, thresholds, flip, out: as lce_bconv2d
 * Covered: C_in a multiple of 32, 3x3 filters over 32 to 192, 256 or 512
 * channels and 5x5 over 32 to 192 or 256, one padding (or a geometry with
 * no padded taps), and an input band (the input rows that the windows of
 * 64 consecutive output pixels read) that fits the LDS of a workgroup.
 * Other requests return LCE_EUNSUPPORTED before anything is launched, and
 * the caller runs lce_bitpack and lce_bconv2d instead.
 * Errors: as lce_bconv2d, plus LCE_EUNSUPPORTED (above) and LCE_EALIGN for
 *         an x that is not 16-byte aligned. */
lce_status lce_quantize_bconv2d(const lce_bconv2d_desc *desc, const float *x,
                                const int32_t *w_packed, const float *multiplier,
                                const float *bias, const float *thresholds,
                                const int32_t *flip, void *out, hipStream_t stream);

/* Number of int32 elements of the zero-padding correction table of `desc`:
 * (KH+1) * KW*(KW+1)/2 * C_out.  Validates the descriptor as lce_bconv2d
 * does.
 * Errors: LCE_EINVAL (null desc/elements, bad field). */
lce_status lce_bconv2d_pad_correction_size(const lce_bconv2d_desc *desc, int64_t *elements);

/* The correction step of zero padding (Section 3.2), prepared once per
 * filter tensor.  With S(co, ky, kx) the sum of the +-1 weights of one tap
 * and I = [x0, x1) one of the NI = KW*(KW+1)/2 non-empty column intervals
 * (numbered by x0, then x1: I = x0*(2*KW - x0 + 1)/2 + x1 - x0 - 1),
 *   pad_correction[(y*NI + I)*C_out + co] = sum over ky < y, kx in I of
 *                                           S(co, ky, kx),   y in [0, KH].
 * The in-image taps of any window form rows [y0, y1) x an interval I, so
 * lce_bconv2d takes their sum as the difference of two entries and removes
 * the padded taps' share.  w_packed as for lce_bconv2d (device, 4-byte aligned);
 * pad_correction: device int32 array of lce_bconv2d_pad_correction_size
 * elements, written asynchronously on `stream`.
 * Errors: LCE_EINVAL (null pointer, bad field, table of 2^31 or more
 *         elements), LCE_EALIGN, LCE_EHIP. */
lce_status lce_bconv2d_pad_correction(const lce_bconv2d_desc *desc, const int32_t *w_packed,
                                      int32_t *pad_correction, hipStream_t stream);

/* Converter-side threshold derivation (Sections 3.1 and 3.2: a binary
 * convolution whose float output only feeds the next layer's binarization
 * can write bits instead, compared against thresholds computed ahead of
 * time).  For each channel it returns thresholds[co] and flip bit co such
 * that, for every clamped accumulator c a convolution with K = k and
 * [clamp_min, clamp_max] can produce,
 *     (c < thresholds[co]) XOR flip[co]  ==  fmaf((float)c, m[co], b[co]) < 0,
 * i.e. lce_bconv2d's bitpacked output with (thresholds, flip) equals
 * lce_bitpack of its float output with (multiplier, bias).  A negative
 * multiplier sets the flip bit; a zero one gives a constant (+-infinity).
 * HOST pointers: multiplier, bias float [c_out] or NULL (= 1.0 / 0.0);
 * thresholds float [c_out] and flip int32 [ceil(c_out/32)] written (pad
 * bits 0).  Synchronous, no GPU work.
 * Errors: LCE_EINVAL (null output, c_out < 1, k outside [1, 2^24],
 *         clamp_min > clamp_max, a non-finite multiplier or bias). */
lce_status lce_fold_thresholds(const float *multiplier, const float *bias, int32_t c_out,
                               int32_t k, int32_t clamp_min, int32_t clamp_max,
                               float *thresholds, int32_t *flip);

/* ---- The same convolution on the matrix cores --------------------------
 *
 * LceBConv2d's dot (Section 3.2) is a dense contraction of +-1 values.  The
 * paper's XOR + POPCOUNT (lce_bconv2d) is how a CPU multiplies them; gfx950's
 * MFMA multiplies 4-bit floats, in which +1.0, -1.0 and 0.0 are exact, and
 * accumulates in fp32, exact for |dot| < 2^24, at eight times the VALU's
 * xor+popcount rate.  lce_bconv2d_mfma computes the identical result from the
 * same bitpacked activations: each bit is widened to a 4-bit +-1.0 only inside
 * the kernel.  The filters are widened once, ahead of time, into a caller-owned
 * buffer (lce_bconv2d_mfma_weights).  Zero padding needs no correction table
 * there: padded locations simply widen to 0.0. */

/* Bytes of the widened filter buffer of `desc` (20 bytes per 32 weights:
 * KH*KW x Cw' words x C_out' filters, Cw' = ceil(C_in/32) rounded up to an
 * even word count or a multiple of 4, C_out' = C_out rounded up to 32; 16
 * bytes widened and 4 bytes packed per word).
 * Errors: LCE_EINVAL (null pointer, bad field). */
lce_status lce_bconv2d_mfma_weights_size(const lce_bconv2d_desc *desc, int64_t *bytes);

/* Widen packed filters w_packed (as for lce_bconv2d, device, 4-byte aligned)
 * into w_fp4 (device, 16-byte aligned, lce_bconv2d_mfma_weights_size bytes),
 * asynchronously on `stream`.  Layout: 16-byte element (t*Cw' + j)*C_out' + co
 * holds word j of tap t of filter co as 32 e2m1 codes (+1.0 = 0x2,
 * -1.0 = 0xA), channel 32j + c in 32-bit word c % 4, nibble c / 4.  Channels
 * past C_in and filters past C_out widen to 0.0.  Then, from byte
 * 16*KH*KW*Cw'*C_out' on, the same elements as packed 32-bit words (bit 1 =
 * -1; channels past C_in, words past Cw and filters past C_out 0): where
 * C_in = 32*Cw', the filter-stationary schedule loads these and widens
 * them itself.  Run once per filter tensor.
 * Errors: LCE_EINVAL, LCE_EALIGN, LCE_EHIP. */
lce_status lce_bconv2d_mfma_weights(const lce_bconv2d_desc *desc, const int32_t *w_packed,
                                    void *w_fp4, hipStream_t stream);

/* LceBConv2d on the matrix cores: arguments, output and every rounding as
 * lce_bconv2d (multiplier/bias for FLOAT32, thresholds and optional flip for
 * BITPACKED), with the widened filters in place of w_packed and either
 * pad_value (no correction table).
 * The work is split by shape between three schedules: filter-stationary
 * (each wave keeps its filters in registers and runs through about one
 * CU's share of pixel blocks; by default up to 36 K steps of 64
 * channels, up to 72 when an instance is forced), K-split
 * (the waves of a workgroup divide K; long K) and pixel-split (the rest).
 * lce_set_tuning can force a schedule, an instance or a tile for tests and
 * tuning; every choice gives the identical output.
 * w_fp4 must be the output of lce_bconv2d_mfma_weights for a descriptor with
 * the same c_in, c_out, kh and kw, 16-byte aligned and at least
 * lce_bconv2d_mfma_weights_size(desc) bytes: the kernels read the widened
 * filters and the packed copy behind them at offsets derived from `desc`
 * (the library cannot see the buffer's size; a smaller one is read past its
 * end).
 * Errors: as lce_bconv2d, plus LCE_EUNSUPPORTED when K = KH*KW*C_in >= 2^24
 * or when the input region a workgroup stages exceeds the LDS of one
 * workgroup (very wide images). */
lce_status lce_bconv2d_mfma(const lce_bconv2d_desc *desc, const int32_t *x_packed,
                            const void *w_fp4, const float *multiplier, const float *bias,
                            const float *thresholds, const int32_t *flip, void *out,
                            hipStream_t stream);

/* LceQuantize followed by the LceBConv2d that consumes it, on the matrix
 * cores in one launch (Section 3.2: the float activation is sign-binarized
 * and bitpacked, then convolved).  The result equals lce_bitpack of x
 * followed by lce_bconv2d_mfma (and so lce_bconv2d) on the packed tensor,
 * bit for bit, with no packed copy written to memory: each workgroup of the
 * filter-stationary or the K-split schedule binarizes the input region its
 * windows read while staging it.
 *   x          float32 [N][H][W][C_in]  (device, 16-byte aligned); the sign
 *              test is lce_bitpack's (x < 0.0f is a 1 bit = -1.0, so -0.0
 *              and NaN give +1.0)
 *   w_fp4, multiplier, bias, thresholds, flip, out: as lce_bconv2d_mfma
 * Covered: C_in a multiple of 32, input below 2 GiB, and the shapes the
 * filter-stationary schedule takes (up to 72 K steps of 64 channels that
 * one of its instances covers with at most 1/8 padding; tried first up to
 * 36 K steps, and beyond where the K split's grid would not fill the CUs)
 * or, from 20 K steps, the K-split one (every 3x3 and 5x5 filter), with an
 * input region per workgroup that fits its LDS.  Other requests (e.g. 1x1
 * filters over few channels) return LCE_EUNSUPPORTED before anything is
 * launched, and the caller runs lce_bitpack and lce_bconv2d_mfma instead.
 * LCE_TUNE_MFMA_SCHEDULE 1 or 2 restricts the choice to that schedule (2
 * then takes any K); 3, the pixel split, has no fused form and is refused.
 * Errors: as lce_bconv2d_mfma, plus LCE_EUNSUPPORTED (above) and LCE_EALIGN
 *         for an x that is not 16-byte aligned. */
lce_status lce_quantize_bconv2d_mfma(const lce_bconv2d_desc *desc, const float *x,
                                     const void *w_fp4, const float *multiplier,
                                     const float *bias, const float *thresholds,
                                     const int32_t *flip, void *out, hipStream_t stream);

/* LceBMaxPool2d (Section 3.2): max pooling of +-1 activations held as
 * bits.  Since max(sign(x)) = sign(max(x)), a max pooling that feeds a
 * binarized layer can run after the binarization, on the packed tensor,
 * where the maximum of +-1 values is the bitwise AND of the window's words
 * (bit 1 = -1.0 survives only if every value in the window is -1).
 * Locations outside the image take no part (TensorFlow max pooling).  The
 * window geometry follows lce_padding like the convolution's. */
typedef struct {
    int32_t n, h, w, channels;     /* input, NHWC bitpacked, >= 1             */
    int32_t kh, kw;                /* window, >= 1                            */
    int32_t stride_h, stride_w;    /* >= 1                                    */
    int32_t padding;               /* lce_padding                             */
} lce_bmaxpool2d_desc;

/* Output height/width of `desc`.
 * Errors: LCE_EINVAL (null pointer, bad field, no output). */
lce_status lce_bmaxpool2d_out_shape(const lce_bmaxpool2d_desc *desc, int32_t *oh, int32_t *ow);

/*   x_packed int32 [N][H][W][ceil(channels/32)]    (device)
 *   out      int32 [N][OH][OW][ceil(channels/32)]  (device); pad bits 0
 * Pointers 4-byte aligned (16-byte alignment and a word count that is a
 * multiple of 4 take the widest loads).
 * Errors: LCE_EINVAL (null pointer, bad field, no output, a tensor of 2^31
 *         or more words), LCE_EALIGN, LCE_EHIP. */
lce_status lce_bmaxpool2d(const lce_bmaxpool2d_desc *desc, const int32_t *x_packed,
                          int32_t *out, hipStream_t stream);

/* LceDequantize (Section 3.2): bitpacked x_packed[rows][ceil(channels/32)]
 * back to float out[rows][channels]: -1.0f where the bit is 1, +1.0f where
 * it is 0 (the inverse of lce_bitpack's sign binarization on +-1 data).
 * rows == 0 is a no-op (pointers may then be NULL).  Pointers 4-byte
 * aligned (a channel count that is a multiple of 32 with out 16-byte aligned
 * takes the widest stores).
 * Errors: LCE_EINVAL (null pointer, rows < 0, channels < 1), LCE_EALIGN,
 *         LCE_EHIP. */
lce_status lce_dequantize(const int32_t *x_packed, float *out, int64_t rows, int32_t channels,
                          hipStream_t stream);

/* ---- Schedule overrides, for tests and tuning ----------------------------
 *
 * Every convolution picks its work split by itself.  These process-wide
 * overrides force one instead; each choice gives the identical output, only
 * the speed changes.  0 (the initial value of every key) restores the
 * library's own choice.  Callers are tests, benchmarks and tuning scripts,
 * not production code.  Values are read once per launch with atomic loads,
 * so setting them while other threads launch is safe (a launch sees either
 * the old or the new value).  An out-of-range value falls back to the
 * automatic choice where the key's comment says so. */
typedef enum {
    LCE_TUNE_XOR_NB = 0,          /* lce_bconv2d: blocks of 8 filters per wave, 1..4    */
    LCE_TUNE_XOR_KS = 1,          /* lce_bconv2d: waves sharing a block's K range 1/2/4 */
    LCE_TUNE_MFMA_SCHEDULE = 2,   /* lce_bconv2d_mfma and lce_quantize_bconv2d_mfma:
                                     1 filter-stationary (where an instance fits),
                                     2 K split, 3 pixel split (not fused)               */
    LCE_TUNE_MFMA_FS_KS = 3,      /* filter-stationary instance: K steps per wave       */
    LCE_TUNE_MFMA_FS_S = 4,       /* filter-stationary instance: waves per filter block */
    LCE_TUNE_MFMA_FS_WPC = 5,     /* filter-stationary grid: 1 or 2 workgroups per CU   */
    LCE_TUNE_MFMA_FS_PAD = 6,     /* -1: no LDS claim that spreads workgroups over CUs  */
    LCE_TUNE_MFMA_PACKED = 7,     /* -1: load widened filters where packed ones would do */
    LCE_TUNE_MFMA_TILE_M = 8,     /* K-split / pixel-split tile: 32-pixel blocks        */
    LCE_TUNE_MFMA_TILE_N = 9,     /* K-split / pixel-split tile: 32-filter blocks       */
    LCE_TUNE_MFMA_FS_WINDOW = 10, /* -1: filter-stationary workgroups stage whole padded
                                     rows, also where a share's window of columns would do */
    LCE_TUNE_COUNT = 11
} lce_tuning_key;

/* Set override `key` to `value` (0 = automatic).
 * Errors: LCE_EINVAL (unknown key). */
lce_status lce_set_tuning(int32_t key, int32_t value);

/* Current value of override `key` (0 for an unknown key). */
int32_t lce_get_tuning(int32_t key);

/* Message describing the last error on the calling thread ("" if none). */
const char *lce_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* LCE_H_ */
