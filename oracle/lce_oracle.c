/*
 * CPU oracle for the bitpacked binary 2-D convolution of Larq Compute Engine
 * (arXiv 2011.09398, Section 3.2 "Operator implementations").
 *
 * TEST INFRASTRUCTURE.  Only the tests, the smoke check and the benchmark's
 * CPU-baseline leg load this library.  It shares no code with the HIP path
 * and must never be used as a fallback for it.
 *
 * Everything here is the plain definition of what the method computes:
 *   - binarization to +-1 values held as int8 (never bit tricks),
 *   - a naive seven-deep cross-correlation over +-1 integers with +1 padding,
 *   - the output transform written out in fp64 (float output) or as an exact
 *     comparison against the threshold (bitpacked output).
 * The XOR/POPCOUNT formulation is deliberately absent: the method reaches
 * exactly this integer result, faster (Section 1; Section 3.2, LceBConv2d).
 *
 * Readings of points the paper leaves open (each one is listed with its
 * justification in the design notes):
 *   - sign: a value is -1 iff x < 0 (so -0.0 and NaN binarize to +1);
 *   - packing: channel c goes to word c/32, bit c%32; unused bits are 0;
 *   - SAME padding follows TensorFlow (extra row/column at bottom/right);
 *   - the fused activation is an integer clamp of the accumulator;
 *   - bitpacked output bit is 1 (meaning -1) iff clamp(dot) < threshold.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

int oracle_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

void oracle_set_num_threads(int n) {
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/*
 * Output size and leading pad of one spatial dimension.
 * SAME:  out = ceil(in / s); total pad = max((out-1)*s + k - in, 0);
 *        the leading side gets floor(total/2), the trailing side the rest.
 * VALID: out = floor((in - k) / s) + 1, no padding.
 * Returns 0 on success, -1 when the shape has no output.
 */
int oracle_out_size(int in, int k, int s, int same, int *out, int *pad_before) {
    if (in < 1 || k < 1 || s < 1) return -1;
    if (same) {
        int o = (in + s - 1) / s;
        int total = (o - 1) * s + k - in;
        if (total < 0) total = 0;
        *out = o;
        *pad_before = total / 2;
        return 0;
    }
    if (in < k) return -1;
    *out = (in - k) / s + 1;
    *pad_before = 0;
    return 0;
}

/* Binarization (LceQuantize, Section 3.2): -1 iff x < 0, else +1. */
void oracle_binarize(const float *x, int64_t count, int8_t *s) {
    for (int64_t i = 0; i < count; ++i) s[i] = (x[i] < 0.0f) ? (int8_t)-1 : (int8_t)1;
}

/*
 * Bitpacking of +-1 values along the innermost axis (LceQuantize): a 0 bit
 * stands for +1 and a 1 bit for -1; the channel count is padded up to a
 * multiple of 32 with 0 bits.
 */
void oracle_pack(const int8_t *s, int64_t rows, int channels, uint32_t *words) {
    int cw = (channels + 31) / 32;
    for (int64_t r = 0; r < rows; ++r) {
        for (int j = 0; j < cw; ++j) {
            uint32_t word = 0;
            for (int b = 0; b < 32; ++b) {
                int c = j * 32 + b;
                if (c < channels && s[r * channels + c] == -1) word |= (uint32_t)1 << b;
            }
            words[r * cw + j] = word;
        }
    }
}

/* The inverse of oracle_pack (LceDequantize's meaning of a bit). */
void oracle_unpack(const uint32_t *words, int64_t rows, int channels, int8_t *s) {
    int cw = (channels + 31) / 32;
    for (int64_t r = 0; r < rows; ++r) {
        for (int c = 0; c < channels; ++c) {
            uint32_t bit = (words[r * cw + c / 32] >> (c % 32)) & 1u;
            s[r * channels + c] = bit ? (int8_t)-1 : (int8_t)1;
        }
    }
}

/*
 * The binary convolution as a plain +-1 integer cross-correlation
 * (LceBConv2d, Section 3.2): for every output pixel and filter,
 *     dot = sum over ky, kx, ci of A(iy, ix, ci) * W(co, ky, kx, ci),
 * with iy = oy*sh - pad_top + ky, ix = ox*sw - pad_left + kx, and A = +1 at
 * every location outside the image ("one-padding": the padded bits are 0,
 * which stand for +1).
 *   a   : int8 +-1, NHWC [n][h][w][c]
 *   wt  : int8 +-1, OHWI [cout][kh][kw][c]
 *   dot : int32, NHWC [n][oh][ow][cout]
 * Returns 0, or -1 for a shape with no output.
 */
int oracle_conv_dot_padded(const int8_t *a, int n, int h, int w, int c,
                           const int8_t *wt, int cout, int kh, int kw,
                           int sh, int sw, int same, int pad, int32_t *dot);

int oracle_conv_dot(const int8_t *a, int n, int h, int w, int c,
                    const int8_t *wt, int cout, int kh, int kw,
                    int sh, int sw, int same, int32_t *dot) {
    return oracle_conv_dot_padded(a, n, h, w, c, wt, cout, kh, kw, sh, sw, same, 1, dot);
}

/*
 * The same cross-correlation with an explicit value at padded locations:
 * pad = 1 is the one-padding above; pad = 0 is TensorFlow's zero-padding,
 * which LCE also supports at the cost of a correction step (Section 3.2).
 */
int oracle_conv_dot_padded(const int8_t *a, int n, int h, int w, int c,
                           const int8_t *wt, int cout, int kh, int kw,
                           int sh, int sw, int same, int pad, int32_t *dot) {
    int oh, ow, pt, pl;
    if (oracle_out_size(h, kh, sh, same, &oh, &pt) != 0) return -1;
    if (oracle_out_size(w, kw, sw, same, &ow, &pl) != 0) return -1;
    int64_t rows = (int64_t)n * oh;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t r = 0; r < rows; ++r) {
        int b = (int)(r / oh);
        int oy = (int)(r % oh);
        for (int ox = 0; ox < ow; ++ox) {
            for (int co = 0; co < cout; ++co) {
                int32_t acc = 0;
                for (int ky = 0; ky < kh; ++ky) {
                    for (int kx = 0; kx < kw; ++kx) {
                        int iy = oy * sh - pt + ky;
                        int ix = ox * sw - pl + kx;
                        int inside = iy >= 0 && iy < h && ix >= 0 && ix < w;
                        const int8_t *wrow = wt + (((int64_t)co * kh + ky) * kw + kx) * c;
                        const int8_t *arow =
                            inside ? a + (((int64_t)b * h + iy) * w + ix) * c : NULL;
                        for (int ci = 0; ci < c; ++ci) {
                            int32_t av = inside ? arow[ci] : pad;
                            acc += av * (int32_t)wrow[ci];
                        }
                    }
                }
                dot[((r * ow) + ox) * (int64_t)cout + co] = acc;
            }
        }
    }
    return 0;
}

/* Fused activation on the integer accumulator: min(max(dot, lo), hi). */
void oracle_clamp(const int32_t *dot, int64_t count, int32_t lo, int32_t hi, int32_t *out) {
    for (int64_t i = 0; i < count; ++i) {
        int32_t v = dot[i];
        if (v < lo) v = lo;
        if (v > hi) v = hi;
        out[i] = v;
    }
}

/*
 * Float output transform: the clamped accumulator converted to a real value,
 * times the per-channel multiplier, plus the per-channel bias, in fp64.
 * mult == NULL means 1, bias == NULL means 0.
 */
void oracle_out_float(const int32_t *c, int64_t m, int cout,
                      const float *mult, const float *bias, double *y) {
    for (int64_t i = 0; i < m; ++i) {
        for (int co = 0; co < cout; ++co) {
            double mm = mult ? (double)mult[co] : 1.0;
            double bb = bias ? (double)bias[co] : 0.0;
            y[i * cout + co] = (double)c[i * cout + co] * mm + bb;
        }
    }
}

/*
 * Bitpacked output transform: output value -1 (bit 1) iff the clamped
 * accumulator is below the channel's threshold, compared exactly (an int32
 * and a float32 are both exact in fp64); NaN thresholds compare false.
 * The results are packed exactly as oracle_pack packs +-1 values.
 */
void oracle_out_bits(const int32_t *c, int64_t m, int cout, const float *thr, uint32_t *words) {
    int cw = (cout + 31) / 32;
    for (int64_t i = 0; i < m; ++i) {
        for (int j = 0; j < cw; ++j) words[i * cw + j] = 0;
        for (int co = 0; co < cout; ++co) {
            if ((double)c[i * cout + co] < (double)thr[co])
                words[i * cw + co / 32] |= (uint32_t)1 << (co % 32);
        }
    }
}

/*
 * Binarized max pooling (LceBMaxPool2d, Section 3.2): the maximum of +-1
 * values over each window, i.e. +1 if any value in the window is +1.
 * Locations outside the image do not take part (TensorFlow max pooling).
 *   a   : int8 +-1, NHWC [n][h][w][c]
 *   out : int8 +-1, NHWC [n][oh][ow][c]
 * Returns 0, or -1 for a shape with no output.
 */
int oracle_bmaxpool(const int8_t *a, int n, int h, int w, int c, int kh, int kw,
                    int sh, int sw, int same, int8_t *out) {
    int oh, ow, pt, pl;
    if (oracle_out_size(h, kh, sh, same, &oh, &pt) != 0) return -1;
    if (oracle_out_size(w, kw, sw, same, &ow, &pl) != 0) return -1;
    for (int b = 0; b < n; ++b)
        for (int oy = 0; oy < oh; ++oy)
            for (int ox = 0; ox < ow; ++ox)
                for (int ci = 0; ci < c; ++ci) {
                    int best = -2;   /* below both values: no valid location seen yet */
                    for (int ky = 0; ky < kh; ++ky)
                        for (int kx = 0; kx < kw; ++kx) {
                            int iy = oy * sh - pt + ky, ix = ox * sw - pl + kx;
                            if (iy < 0 || iy >= h || ix < 0 || ix >= w) continue;
                            int v = a[(((int64_t)b * h + iy) * w + ix) * c + ci];
                            if (v > best) best = v;
                        }
                    out[(((int64_t)b * oh + oy) * ow + ox) * c + ci] = (int8_t)best;
                }
    return 0;
}

/*
 * The next layer's binarization of a float-output transform (Section 3.1):
 * bit(c) = 1 iff fmaf((float)c, mult, bias) < 0.  For integer c and float
 * mult, bias, the exact value c*mult + bias is a multiple of 2^-149, so it is
 * never rounded to -0.0 and its sign decides; c*mult is exact in fp64 for
 * |c| < 2^24 and fp64 rounding of the sum keeps a nonzero sign.
 */
void oracle_sign_of_affine(const int32_t *c, int64_t count, float mult, float bias,
                           uint8_t *bits) {
    for (int64_t i = 0; i < count; ++i) {
        double x = (double)c[i] * (double)mult + (double)bias;
        bits[i] = (uint8_t)(x < 0.0);
    }
}
