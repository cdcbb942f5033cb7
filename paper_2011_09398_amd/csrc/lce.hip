// C ABI of the MI355X bitpacked binary convolution (declared in include/lce.h):
// host-side validation, geometry and kernel dispatch.  No allocation, no
// synchronization: every launch goes on the caller's stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <climits>
#include <cmath>
#include <cstdarg>
#include <cstdlib>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <numeric>
#include <string>

#include "lce.h"
#include "bitpack.hpp"
#include "bconv.hpp"
#include "pool.hpp"
#include "bconv_mfma.hpp"
#include "launch.hpp"

// Kernels that run once per filter tensor (not on the timed path).
namespace lce {

// The zero-padding table of one filter tensor:
//   table[(y*NI + I)*Cout + co] = sum over ky < y, kx in I of S(co, ky, kx),
//   S(co, ky, kx) = C_in - 2*popcount(W[co][ky][kx][:])  (the sum of the tap's
//   +-1 weights; pad bits are 0 and count nothing),
// for y in [0, KH] and the NI = KW(KW+1)/2 column intervals I = [x0, x1).
// One thread per filter; a filter tensor needs it once.
__device__ inline int tap_sum(const uint32_t *w, int co, int ky, int kx, int kh, int kw, int cw,
                              int cin) {
    const uint32_t *wt = w + (((size_t)co * kh + ky) * kw + kx) * cw;
    int pc = 0;
    for (int j = 0; j < cw; ++j) pc += __builtin_popcount(wt[j]);
    return cin - 2 * pc;
}

__global__ __launch_bounds__(256) void pad_table_kernel(const uint32_t *__restrict__ w,
                                                        int32_t *__restrict__ table, int cout,
                                                        int kh, int kw, int cw, int cin) {
    const int co = blockIdx.x * blockDim.x + threadIdx.x;
    if (co >= cout) return;
    const size_t ni = (size_t)interval_count(kw);
    for (size_t i = 0; i < ni; ++i) table[i * cout + co] = 0;        // y = 0
    for (int y = 1; y <= kh; ++y) {
        for (int x0 = 0; x0 < kw; ++x0) {
            int run = 0;
            for (int x1 = x0 + 1; x1 <= kw; ++x1) {
                run += tap_sum(w, co, y - 1, x1 - 1, kh, kw, cw, cin);
                const size_t i = (size_t)interval_index(x0, x1, kw);
                table[((size_t)y * ni + i) * cout + co] =
                    table[((size_t)(y - 1) * ni + i) * cout + co] + run;
            }
        }
    }
}

// Filters widened once per filter tensor into the B layout:
//   wexp[(t*CwE + j)*CoutP + co] = 32 e2m1 codes of word j of tap t of
//   filter co, in the order of widen_word (channel c of the word in 32-bit
//   word c % 4, nibble c / 4); channels past C_in, words past Cw and filters
//   past Cout are 0.0 (they then add nothing to any dot);
//   wpk[same index] = the packed word itself (bits of channels past C_in
//   cleared; words past Cw and filters past Cout 0), for kernels that
//   widen the filters themselves where every channel is valid.
__global__ __launch_bounds__(256) void mfma_expand_weights_kernel(const uint32_t *__restrict__ w,
                                                                  u32x4 *__restrict__ wexp,
                                                                  uint32_t *__restrict__ wpk,
                                                                  int cout, int coutp, int taps,
                                                                  int cw, int cwe, int cin) {
    const int64_t total = (int64_t)taps * cwe * coutp;
    for (int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * 256) {
        const int64_t k = idx / coutp;
        const int co = (int)(idx - k * coutp);
        const int t = (int)(k / cwe), j = (int)(k - (int64_t)t * cwe);
        u32x4 o = {0u, 0u, 0u, 0u};
        uint32_t packed = 0u;
        if (co < cout && j < cw) {
            const uint32_t bits = w[((size_t)co * taps + t) * cw + j];
            const int nvalid = min(32, cin - 32 * j);
            const uint32_t valid = nvalid >= 32 ? 0xFFFFFFFFu : (1u << nvalid) - 1u;
            o = widen_word(bits, kFp4PlusOne) & widen_valid_mask(valid);
            packed = bits & valid;
        }
        wexp[idx] = o;
        wpk[idx] = packed;
    }
}

}  // namespace lce

namespace {

thread_local std::string g_last_error;

lce_status fail(lce_status st, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return st;
}

lce_status ok() {
    g_last_error.clear();
    return LCE_OK;
}

lce_status check_launch(const char *what) {
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(LCE_EHIP, "%s: %s", what, hipGetErrorString(e));
    return ok();
}

bool aligned(const void *p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

int packed_words(int channels) { return (channels + 31) / 32; }

// TensorFlow SAME/VALID output size, leading pad and total pad of one
// dimension.
bool out_dim(int in, int k, int s, int padding, int *out, int *pad_before, long *pad_total) {
    if (padding == LCE_PADDING_SAME) {
        const int o = in / s + (in % s != 0);
        long total = (long)(o - 1) * s + k - in;
        if (total < 0) total = 0;
        *out = o;
        *pad_before = (int)(total / 2);
        *pad_total = total;
        return true;
    }
    if (in < k) return false;
    *out = (in - k) / s + 1;
    *pad_before = 0;
    *pad_total = 0;
    return true;
}

struct Geometry {
    int oh, ow, pt, pl;
    bool pads;   // some window reaches outside the image
};

// Elements of the zero-padding table: (KH+1) row prefixes x KW(KW+1)/2
// column intervals x C_out.
int64_t table_elements(const lce_bconv2d_desc &d) {
    return (int64_t)(d.kh + 1) * ((int64_t)d.kw * (d.kw + 1) / 2) * d.c_out;
}

// Zero padding changes the result only where some window reaches outside
// the image; there it needs the correction table.
bool zero_padded(const lce_bconv2d_desc &d, const Geometry &g) {
    return d.pad_value == LCE_PAD_ZERO && g.pads;
}

lce_status validate_desc(const lce_bconv2d_desc *d, Geometry *g) {
    if (!d) return fail(LCE_EINVAL, "desc is NULL");
    if (d->n < 1 || d->h < 1 || d->w < 1 || d->c_in < 1)
        return fail(LCE_EINVAL, "input dims must be >= 1 (n=%d h=%d w=%d c_in=%d)", d->n, d->h,
                    d->w, d->c_in);
    if (d->c_out < 1 || d->kh < 1 || d->kw < 1)
        return fail(LCE_EINVAL, "filter dims must be >= 1 (c_out=%d kh=%d kw=%d)", d->c_out,
                    d->kh, d->kw);
    if (d->stride_h < 1 || d->stride_w < 1)
        return fail(LCE_EINVAL, "strides must be >= 1 (%d, %d)", d->stride_h, d->stride_w);
    if (d->padding != LCE_PADDING_VALID && d->padding != LCE_PADDING_SAME)
        return fail(LCE_EINVAL, "unknown padding %d", d->padding);
    if (d->pad_value != LCE_PAD_ONE && d->pad_value != LCE_PAD_ZERO)
        return fail(LCE_EINVAL, "unknown pad_value %d", d->pad_value);
    if (d->out_type != LCE_OUT_FLOAT32 && d->out_type != LCE_OUT_BITPACKED &&
        d->out_type != LCE_OUT_INT32)
        return fail(LCE_EINVAL, "unknown out_type %d", d->out_type);
    if (d->clamp_min > d->clamp_max)
        return fail(LCE_EINVAL, "clamp_min %d > clamp_max %d", d->clamp_min, d->clamp_max);
    long th = 0, tw = 0;
    if (!out_dim(d->h, d->kh, d->stride_h, d->padding, &g->oh, &g->pt, &th) ||
        !out_dim(d->w, d->kw, d->stride_w, d->padding, &g->ow, &g->pl, &tw))
        return fail(LCE_EINVAL, "VALID convolution with a %dx%d filter has no output on %dx%d",
                    d->kh, d->kw, d->h, d->w);
    g->pads = th > 0 || tw > 0;
    const int64_t cw = packed_words(d->c_in);
    const int64_t m = (int64_t)d->n * g->oh * g->ow;
    const int64_t x_words = (int64_t)d->n * d->h * d->w * cw;
    const int64_t w_words = (int64_t)d->c_out * d->kh * d->kw * cw;
    const int64_t out_elems = m * (d->out_type == LCE_OUT_BITPACKED ? packed_words(d->c_out)
                                                                    : d->c_out);
    const int64_t k = (int64_t)d->kh * d->kw * d->c_in;
    const int64_t lim = INT32_MAX;
    if (m > lim - lce::kPix || x_words > lim || w_words > lim || out_elems > lim || k > lim / 2)
        return fail(LCE_EINVAL,
                    "tensor too large (pixels %lld, input words %lld, filter words %lld, "
                    "output elements %lld, K %lld; each must stay below 2^31)",
                    (long long)m, (long long)x_words, (long long)w_words, (long long)out_elems,
                    (long long)k);
    if (d->c_out > (1 << 20)) return fail(LCE_EINVAL, "c_out %d exceeds 2^20", d->c_out);
    const int64_t table = table_elements(*d);
    if (zero_padded(*d, *g) && (k >= (1 << 29) || table > lim))
        return fail(LCE_EINVAL,
                    "zero padding needs K < 2^29 and a correction table below 2^31 elements "
                    "(K %lld, table %lld)", (long long)k, (long long)table);
    return ok();
}

using lce::BconvParams;

// The launch parameters of an XOR/POPCOUNT convolution that depend only on
// the descriptor, the filters and the output transform (the input pointer,
// the zero-padding table and the schedule are set by the caller).
BconvParams bconv_params(const lce_bconv2d_desc &d, const Geometry &g, const int32_t *w_packed,
                         const float *multiplier, const float *bias, const float *thresholds,
                         const int32_t *flip, void *out) {
    BconvParams p{};
    p.w = reinterpret_cast<const uint32_t *>(w_packed);
    p.mult = d.out_type == LCE_OUT_FLOAT32 ? multiplier : nullptr;
    p.bias = d.out_type == LCE_OUT_FLOAT32 ? bias : nullptr;
    p.thr = thresholds;
    p.flip = d.out_type == LCE_OUT_BITPACKED ? reinterpret_cast<const uint32_t *>(flip) : nullptr;
    p.out = out;
    p.n = d.n; p.h = d.h; p.wd = d.w; p.cw = packed_words(d.c_in);
    p.oh = g.oh; p.ow = g.ow; p.cout = d.c_out; p.cwo = packed_words(d.c_out);
    p.kh = d.kh; p.kw = d.kw; p.sh = d.stride_h; p.sw = d.stride_w; p.pt = g.pt; p.pl = g.pl;
    p.kwords = d.kh * d.kw * p.cw;
    p.k = d.kh * d.kw * d.c_in;
    p.lo = d.clamp_min; p.hi = d.clamp_max;
    p.m = d.n * g.oh * g.ow;
    p.out_vec4 = aligned(out, 16) ? 1 : 0;
    p.div_ohw = lce::make_fastdiv((uint32_t)(g.oh * g.ow));
    p.div_ow = lce::make_fastdiv((uint32_t)g.ow);
    return p;
}

// The quantize-fused convolution: the tallest band of input rows that the
// windows of one workgroup's 64 consecutive output pixels read (global rows
// n*H + y, first in-image row of the first pixel to last of the last).  A
// block's band depends only on its first pixel's offset within the image (a
// block cut short by the end of the batch is no taller than a full one at
// the same offset), and the offset repeats every ohw / gcd(64, ohw) blocks,
// so one such period covers every block.
int64_t quant_band_rows(const BconvParams &p) {
    const int64_t ohw = (int64_t)p.oh * p.ow;
    const int64_t blocks = ((int64_t)p.m + lce::kPix - 1) / lce::kPix;
    const int64_t period = ohw / std::gcd<int64_t>(lce::kPix, ohw);
    int64_t tallest = 0;
    for (int64_t b = 0; b < std::min(blocks, period); ++b) {
        const int64_t ma = b * lce::kPix, mb = std::min(ma + lce::kPix - 1, (int64_t)p.m - 1);
        const int64_t ia = ma / ohw, oya = (ma - ia * ohw) / p.ow;
        const int64_t ib = mb / ohw, oyb = (mb - ib * ohw) / p.ow;
        const int64_t first = ia * p.h + std::max<int64_t>(0, oya * p.sh - p.pt);
        const int64_t last =
            ib * p.h + std::min<int64_t>(p.h - 1, oyb * p.sh - p.pt + p.kh - 1);
        tallest = std::max(tallest, last - first + 1);
    }
    return tallest;
}

// Why lce_quantize_bconv2d does not cover a valid descriptor, or NULL.
const char *quant_unsupported(const lce_bconv2d_desc &d, const Geometry &g) {
    if (zero_padded(d, g)) return "zero padding is not fused";
    if (d.c_in % 32 != 0) return "c_in is not a multiple of 32";
    if (!lce::has_quant_instance(d.c_in / 32, d.kh, d.kw))
        return "no fused instance for this filter size and channel count";
    return nullptr;
}

template <int CW, int KH, int KW, int OUT, bool PADZ>
void launch_static(const BconvParams &p0, dim3 grid, hipStream_t s, int vec) {
    // zero padding: the correction table's rows in dynamic LDS
    const size_t lds =
        PADZ ? (size_t)lce::table_lds_words((KH + 1) * lce::interval_count(KW), p0.fwg) *
                   sizeof(int32_t)
             : 0;
    // tiles renumbered filter-major per XCD where the filters outweigh the
    // input (and the tile count fits the kernel's 32-bit tile arithmetic)
    BconvParams p = p0;
    const double filter_bytes = 4.0 * p.cout * p.kwords;
    const double input_bytes = 4.0 * p.n * p.h * p.wd * p.cw;
    const int64_t tiles = (int64_t)grid.x * grid.y;
    p.tiles = filter_bytes > input_bytes && tiles <= INT32_MAX ? (int)tiles : 0;
    p.div_tile = lce::make_fastdiv(grid.x);
    if (vec == 4 && CW % 4 == 0)
        hipLaunchKernelGGL(
            (lce::bconv2d_static_kernel<CW, KH, KW, (CW % 4 == 0 ? 4 : 1), OUT, PADZ>), grid,
            dim3(lce::kThreads), lds, s, p);
    else if (vec >= 2 && CW % 2 == 0)
        hipLaunchKernelGGL(
            (lce::bconv2d_static_kernel<CW, KH, KW, (CW % 2 == 0 ? 2 : 1), OUT, PADZ>), grid,
            dim3(lce::kThreads), lds, s, p);
    else
        hipLaunchKernelGGL((lce::bconv2d_static_kernel<CW, KH, KW, 1, OUT, PADZ>), grid,
                           dim3(lce::kThreads), lds, s, p);
}

template <int OUT, bool PADZ>
void launch_generic(const BconvParams &p, dim3 grid, hipStream_t s) {
    const size_t lds = (size_t)lce::kPix * p.rs * sizeof(uint32_t);
    hipLaunchKernelGGL((lce::bconv2d_generic_kernel<OUT, PADZ>), grid, dim3(lce::kThreads), lds,
                       s, p);
}

// Shapes with a specialized instance: 3x3 and 5x5 filters over the word
// counts of 32 to 512 (3x3) or 256 (5x5) channels that networks and the
// paper's convolution sweep use; every other shape runs the generic kernel.
bool has_static(int cw, int kh, int kw) {
    if (kh == 3 && kw == 3)
        return (cw >= 1 && cw <= 6) || cw == 8 || cw == 16;
    if (kh == 5 && kw == 5)
        return (cw >= 1 && cw <= 6) || cw == 8;
    return false;
}

// The shape-specialized kernels stage the input through buffer loads (byte
// offsets below 2^31); a larger input runs the generic kernel.
bool input_fits_buffer(const BconvParams &p) {
    return (int64_t)p.n * p.h * p.wd * p.cw * 4 < (int64_t(1) << 31);
}

template <int OUT, bool PADZ>
void dispatch(const BconvParams &p, dim3 grid, hipStream_t s, int vec) {
    if (!input_fits_buffer(p)) {
        launch_generic<OUT, PADZ>(p, grid, s);
        return;
    }
    if (p.kh == 3 && p.kw == 3) {
        switch (p.cw) {
            case 1: launch_static<1, 3, 3, OUT, PADZ>(p, grid, s, vec); return;
            case 2: launch_static<2, 3, 3, OUT, PADZ>(p, grid, s, vec); return;
            case 3: launch_static<3, 3, 3, OUT, PADZ>(p, grid, s, vec); return;
            case 4: launch_static<4, 3, 3, OUT, PADZ>(p, grid, s, vec); return;
            case 5: launch_static<5, 3, 3, OUT, PADZ>(p, grid, s, vec); return;
            case 6: launch_static<6, 3, 3, OUT, PADZ>(p, grid, s, vec); return;
            case 8: launch_static<8, 3, 3, OUT, PADZ>(p, grid, s, vec); return;
            case 16: launch_static<16, 3, 3, OUT, PADZ>(p, grid, s, vec); return;
            default: break;
        }
    } else if (p.kh == 5 && p.kw == 5) {
        switch (p.cw) {
            case 1: launch_static<1, 5, 5, OUT, PADZ>(p, grid, s, vec); return;
            case 2: launch_static<2, 5, 5, OUT, PADZ>(p, grid, s, vec); return;
            case 3: launch_static<3, 5, 5, OUT, PADZ>(p, grid, s, vec); return;
            case 4: launch_static<4, 5, 5, OUT, PADZ>(p, grid, s, vec); return;
            case 5: launch_static<5, 5, 5, OUT, PADZ>(p, grid, s, vec); return;
            case 6: launch_static<6, 5, 5, OUT, PADZ>(p, grid, s, vec); return;
            case 8: launch_static<8, 5, 5, OUT, PADZ>(p, grid, s, vec); return;
            default: break;
        }
    }
    launch_generic<OUT, PADZ>(p, grid, s);
}

template <int OUT>
void dispatch(const BconvParams &p, dim3 grid, hipStream_t s, int vec, bool padz) {
    if (padz)
        dispatch<OUT, true>(p, grid, s, vec);
    else
        dispatch<OUT, false>(p, grid, s, vec);
}

// Schedule overrides (lce_set_tuning): 0 = the library's own choice.  Each
// launch reads every value it uses once, with a relaxed atomic load, so a
// concurrent lce_set_tuning is never a data race (a launch sees the old or
// the new value).
std::atomic<int32_t> g_tuning[LCE_TUNE_COUNT];

int tuning(lce_tuning_key key) { return g_tuning[key].load(std::memory_order_relaxed); }

// A device attribute, cached per device.  The cache entries are atomics: two
// threads making their first launch together both query the attribute and
// store the same value.
template <hipDeviceAttribute_t ATTR>
int device_attribute(int fallback) {
    static std::atomic<int> cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return fallback;
    int v = cache[dev].load(std::memory_order_relaxed);
    if (v == 0) {
        if (hipDeviceGetAttribute(&v, ATTR, dev) != hipSuccess || v <= 0) v = fallback;
        cache[dev].store(v, std::memory_order_relaxed);
    }
    return v;
}

// SIMDs of the current device (4 per compute unit).
int device_simds() { return 4 * device_attribute<hipDeviceAttributeMultiprocessorCount>(256); }

// Work schedule of the shape-specialized kernel.  A unit is 64 pixels x 8
// filters x the whole K range.  Each schedule (nb filter blocks per wave, or
// K split over ks waves) is priced as the VALU instructions on the busiest
// SIMD: ceil(waves / SIMDs) x instructions per wave, where a wave issues
// 16 * Kw * nb / ks xor/popcount instructions plus ~105 + Kw/2 for staging
// and set-up, ~35 per extra block and ~20 for a K-split reduction (counts
// from the measured instruction mix).  Schedules with fewer than 2 waves per
// SIMD are only used when nothing else is possible: a lone wave cannot hide
// its own memory latency.  The xor_nb / xor_ks tuning keys override the
// choice.
void choose_schedule(BconvParams &p, int filters) {
    const long pix_blocks = (p.m + lce::kPix - 1) / lce::kPix;
    const long units = pix_blocks * ((filters + lce::kRN - 1) / lce::kRN);
    const long simds = device_simds();
    static const int kOptions[][2] = {{1, 1}, {2, 1}, {4, 1}, {1, 2}, {1, 4}};
    // key: occupied schedules first; among them the lowest cost, otherwise
    // the most waves.
    int nb = 1, ks = 1;
    bool have = false, best_occupied = false;
    double best_key = 0;
    for (const auto &o : kOptions) {
        const int onb = o[0], oks = o[1];
        if (oks > 1 && p.kwords < 4 * oks) continue;
        const long waves = (units * oks + onb - 1) / onb;
        const long rounds = (waves + simds - 1) / simds;
        const double per_wave = 16.0 * p.kwords * onb / oks + 105.0 + 0.5 * p.kwords +
                                35.0 * (onb - 1) + (oks > 1 ? 20.0 : 0.0);
        const bool occupied = waves >= 2 * simds;
        const double key = occupied ? (double)rounds * per_wave : -(double)waves;
        if (!have || (occupied && !best_occupied) ||
            (occupied == best_occupied && key < best_key)) {
            have = true; best_occupied = occupied; best_key = key; nb = onb; ks = oks;
        }
    }
    if (const int t = tuning(LCE_TUNE_XOR_KS)) ks = t;
    if (const int t = tuning(LCE_TUNE_XOR_NB)) nb = t;
    if (ks != 1 && ks != 2 && ks != 4) ks = 1;
    if (ks > 1) nb = 1;
    if (nb < 1) nb = 1;
    if (nb > lce::kMaxNB) nb = lce::kMaxNB;
    p.ks = ks;
    p.nb = nb;
    p.fwg = (lce::kWaves / ks) * nb * lce::kRN;
    p.ksplit = ((p.kwords + ks - 1) / ks + 3) / 4 * 4;
}

lce_status validate_pool(const lce_bmaxpool2d_desc *d, Geometry *g) {
    if (!d) return fail(LCE_EINVAL, "desc is NULL");
    if (d->n < 1 || d->h < 1 || d->w < 1 || d->channels < 1)
        return fail(LCE_EINVAL, "input dims must be >= 1 (n=%d h=%d w=%d channels=%d)", d->n,
                    d->h, d->w, d->channels);
    if (d->kh < 1 || d->kw < 1 || d->stride_h < 1 || d->stride_w < 1)
        return fail(LCE_EINVAL, "window %dx%d and strides (%d, %d) must be >= 1", d->kh, d->kw,
                    d->stride_h, d->stride_w);
    if (d->padding != LCE_PADDING_VALID && d->padding != LCE_PADDING_SAME)
        return fail(LCE_EINVAL, "unknown padding %d", d->padding);
    long th = 0, tw = 0;
    if (!out_dim(d->h, d->kh, d->stride_h, d->padding, &g->oh, &g->pt, &th) ||
        !out_dim(d->w, d->kw, d->stride_w, d->padding, &g->ow, &g->pl, &tw))
        return fail(LCE_EINVAL, "VALID pooling with a %dx%d window has no output on %dx%d",
                    d->kh, d->kw, d->h, d->w);
    g->pads = th > 0 || tw > 0;
    const int64_t cw = packed_words(d->channels);
    const int64_t in_words = (int64_t)d->n * d->h * d->w * cw;
    const int64_t out_words = (int64_t)d->n * g->oh * g->ow * cw;
    if (in_words > INT32_MAX || out_words > INT32_MAX)
        return fail(LCE_EINVAL, "tensor too large (input words %lld, output words %lld; each "
                    "must stay below 2^31)", (long long)in_words, (long long)out_words);
    return ok();
}

template <int VEC>
void launch_pool(const lce::PoolParams &p, hipStream_t s) {
    int64_t blocks = (p.units + lce::kPoolThreads - 1) / lce::kPoolThreads;
    if (blocks > 256 * 16) blocks = 256 * 16;
    const dim3 grid((unsigned)blocks), block(lce::kPoolThreads);
    if (p.kh == 2 && p.kw == 2)
        hipLaunchKernelGGL((lce::bmaxpool_kernel<VEC, 2, 2>), grid, block, 0, s, p);
    else if (p.kh == 3 && p.kw == 3)
        hipLaunchKernelGGL((lce::bmaxpool_kernel<VEC, 3, 3>), grid, block, 0, s, p);
    else
        hipLaunchKernelGGL((lce::bmaxpool_kernel<VEC, 0, 0>), grid, block, 0, s, p);
}

// ---- matrix-core path

// Channel words per LDS chunk (2 or 4; the K step of the MFMA is a word
// pair) and the word count padded to it: the smaller padding wins, 4 on ties.
void mfma_chunk(int cw, int *cc, int *cwe) {
    const int e2 = (cw + 1) / 2 * 2, e4 = (cw + 3) / 4 * 4;
    *cc = e2 < e4 ? 2 : 4;
    *cwe = e2 < e4 ? e2 : e4;
}

int64_t mfma_weight_bytes(const lce_bconv2d_desc &d) {
    int cc, cwe;
    mfma_chunk(packed_words(d.c_in), &cc, &cwe);
    const int64_t coutp = (int64_t)(d.c_out + 31) / 32 * 32;
    return (int64_t)d.kh * d.kw * cwe * coutp * (16 + 4);   // widened, then packed
}

int device_max_lds() { return device_attribute<hipDeviceAttributeMaxSharedMemoryPerBlock>(65536); }

// Stacked padded rows a workgroup of `bm` pixels reads, maximized over the
// workgroups (the span repeats with the image, so one period suffices).
int mfma_tile_rows(const lce::MfmaParams &p, int bm) {
    const int64_t per_img = (int64_t)p.oh * p.ow;
    const int64_t blocks = ((int64_t)p.m + bm - 1) / bm;
    int64_t g = per_img, b = bm;
    while (b) { const int64_t t = g % b; g = b; b = t; }
    const int64_t period = per_img / g;           // blocks until the pattern repeats
    auto row_of = [&](int64_t m) {
        const int64_t img = m / per_img, r = m % per_img;
        return img * p.ph + (r / p.ow) * p.sh;
    };
    int64_t best = 0;
    for (int64_t i = 0; i < std::min(blocks, period + 1); ++i) {
        const int64_t first = i * bm;
        const int64_t last = std::min(first + bm - 1, (int64_t)p.m - 1);
        best = std::max(best, row_of(last) - row_of(first) + p.kh);
    }
    return (int)best;
}

// The filter-stationary step table: A-tile offset of K step s (tap t, word
// pair q), 2q*plane + ky*PW + kx, with the real channels of the word pair,
// min(64, C_in - 64q), in bits 24-31; steps past the last repeat it.
void fill_step_table(lce::MfmaParams &p, const lce_bconv2d_desc &d, int plane, int ksteps) {
    const int cwh = p.cwe / 2;
    for (int s = 0; s < lce::kFsMaxSteps; ++s) {
        const int sc = std::min(s, ksteps - 1);
        const int t = sc / cwh, q = sc % cwh;
        const int vc = std::min(64, std::max(0, d.c_in - 64 * q));
        p.fs_koff[s] = (2 * q * plane + (t / d.kw) * p.pw + t % d.kw) | (vc << 24);
    }
}

// Filter-stationary instances: K steps per wave (KS) and waves sharing a
// filter block (S).
struct FsShape {
    int ks, s;
};
constexpr FsShape kFsShapes[] = {{9, 1}, {18, 1}, {5, 2}, {9, 2}, {18, 2}, {18, 4}};

// LDS of the filter-stationary kernel: every widened word of the region
// (staged through registers), then (S > 1) the partial-sum exchange: two
// buffers x F filter blocks x two pixel blocks x (S-1) partials, 4 KB each;
// then the bounds of the F filter blocks (bitpacked output) and the A-tile
// offset of each pixel's window origin (one int per pixel of the
// workgroup's whole blocks).
// Bytes from the end of the A tile to the bounds (after the exchange).
size_t mfma_fs_thr_offset(FsShape sh) {
    return sh.s > 1 ? (size_t)2 * (4 / sh.s) * 2 * (sh.s - 1) * 4096 : 0;
}

size_t mfma_fs_lds(const lce::MfmaParams &p, FsShape sh, int tile_rows, int width, int pixels) {
    const size_t a = (size_t)p.cwe * tile_rows * width * 16;
    return a + mfma_fs_thr_offset(sh) + (4 / sh.s) * 32 * 4 + (size_t)(pixels + 31) / 32 * 32 * 4;
}

struct FsPlan {
    FsShape shape{0, 0};
    int pixels = 0, tile_rows = 0, wpc = 1;
    int width = 0;          // padded columns each workgroup stages
    bool window = false;    // width < pw: each share's own window of columns
    int64_t groups = 0;
    size_t lds = 0;
};

// Workgroups per CU the filter-stationary grid is sized for.  Two (two
// waves per SIMD, each hiding the other's finishing work and LDS waits
// behind its matrix products) where a wave's filters are few, KS <= 9 and
// S = 1, and one workgroup per CU would still hold more than one pixel
// block (`px1`: its pixels): measured about 1.1x faster on the batch-64
// 56x56x64->128/s2 layer (9 K steps), while where one block per workgroup
// is all there is (batch-1 layers) the second workgroup only adds its
// set-up (56x56x64->64: 3.92 vs 3.53 us).  With KS = 18 the second
// workgroup's filter loads and widening cost more than the overlap gains
// (measured slower on 28x28x128).  Every instance with S = 1 and KS <= 9
// keeps its registers within the 256 per lane that two waves per SIMD
// leave.  The mfma_fs_wpc tuning key (1 or 2) forces it.
int fs_wgs_per_cu(FsShape sh, int64_t px1) {
    const int e = tuning(LCE_TUNE_MFMA_FS_WPC);
    if (e == 1 || e == 2) return e;
    return sh.s == 1 && sh.ks <= 9 && px1 > 32 ? 2 : 1;
}

// Price of the partial-sum exchange of an instance with S > 1, in matrix
// products per workgroup: a fixed part (two barriers, the sums written and
// read back through LDS) plus one product per pixel block.  Calibrated on
// the batch-1 layers of one block per workgroup: (9, 1) beats (5, 2) on
// 56x56x64->64 (3.53 vs 3.68 us) and 56x56x64->128/s2 (3.32 vs 3.42), and
// (9, 2) beats (18, 1) on 28x28x128->128 (3.53 vs 3.74), so the fixed part
// lies between 3 and 8 products.
constexpr int64_t kFsExchangeFixed = 4;

// Whether filter-stationary instance sh takes a layer of `ksteps` K steps:
// its waves cover them with every wave busy and (unless an instance is
// forced through the tuning keys) at most 1/8 of them padding; a forced
// instance or S excludes the others.
bool fs_shape_takes(FsShape sh, int64_t ksteps) {
    const int env_ks = tuning(LCE_TUNE_MFMA_FS_KS), env_s = tuning(LCE_TUNE_MFMA_FS_S);
    if (env_ks && sh.ks != env_ks) return false;
    if (env_s && sh.s != env_s) return false;
    const int cover = sh.ks * sh.s;
    if (cover < ksteps || cover - sh.ks >= ksteps) return false;   // every wave has work
    return (env_ks && env_s) || (cover - ksteps) * 8 <= ksteps;
}

bool fs_any_takes(int64_t ksteps) {
    for (const FsShape &sh : kFsShapes)
        if (fs_shape_takes(sh, ksteps)) return true;
    return false;
}

// The filter-stationary plan of a layer: among the instances whose K steps
// cover the layer's with at most 1/8 padding (any, when forced), the one
// with the fewest matrix products per SIMD (pixel blocks per workgroup x
// KS, plus the exchange, x workgroups per CU), with about wpc workgroups
// per CU: each filter group gets wpc x CUs / filter groups workgroups,
// each an equal share of the pixels.  A share shorter than an output row
// is rounded up to a divisor of OW where that keeps its pixel block count,
// so that every share lies within one output row; each workgroup then
// stages only the (px - 1)*sw + KW padded columns its windows read, not
// whole rows (batch 1: the 56x56x64->128/s2 layer's 4-pixel shares read 9
// of 57 columns), or, where that window is the whole row, KH rows instead
// of the KH + sh of a share across two output rows.  A longer share is
// rounded up to whole output rows where that keeps its block count and
// stages no more rows (batch 16, 28x28x128: 56 pixels over 4 padded rows
// instead of 49 over 5; batch 64, 56x56x64->128/s2: 112 pixels, 3.5 of its
// 4 blocks useful instead of 98 pixels' 3.06, over the same 9 rows, with
// fewer workgroups).  shape.ks == 0: none fits.
FsPlan plan_mfma_fs(const lce::MfmaParams &p, int64_t cus, int blocks32, int ksteps) {
    FsPlan best;
    int64_t best_cost = -1;
    for (const FsShape &sh : kFsShapes) {
        if (!fs_shape_takes(sh, ksteps)) continue;
        const int f = 4 / sh.s;
        const int64_t fgroups = (blocks32 + f - 1) / f;
        const int64_t pg1 = std::max<int64_t>(1, cus / fgroups);
        const int wpc = fs_wgs_per_cu(sh, ((int64_t)p.m + pg1 - 1) / pg1);
        const int64_t pg = std::max<int64_t>(1, cus * wpc / fgroups);
        // (not rounded to whole blocks: the block count is the same, and an
        // exact share often covers whole images or rows, with fewer rows)
        int64_t px = ((int64_t)p.m + pg - 1) / pg;
        if (px > (1 << 20)) continue;
        int width = p.pw;
        int tr = mfma_tile_rows(p, (int)px);
        if (px < p.ow && tuning(LCE_TUNE_MFMA_FS_WINDOW) >= 0) {
            int64_t dv = px;
            while (p.ow % dv) ++dv;                       // (OW itself at the latest)
            const int w = (int)((dv - 1) * p.sw + p.kw);
            const int tr_dv = mfma_tile_rows(p, (int)dv);
            if ((dv + 31) / 32 == (px + 31) / 32 && (w < p.pw || tr_dv < tr)) {
                px = dv;
                width = w;
                tr = tr_dv;
            }
        } else if (px % p.ow && tuning(LCE_TUNE_MFMA_FS_WINDOW) >= 0) {
            // a share of several rows: whole rows where that stages no more
            const int64_t dv = (px + p.ow - 1) / p.ow * p.ow;
            const int tr_dv = mfma_tile_rows(p, (int)dv);
            if ((dv + 31) / 32 == (px + 31) / 32 && tr_dv <= tr) {
                px = dv;
                tr = tr_dv;
            }
        }
        const size_t lds = mfma_fs_lds(p, sh, tr, width, (int)px);
        if (lds > (size_t)device_max_lds()) continue;
        if ((int64_t)tr * width * p.cwe > INT32_MAX / 2) continue;
        const int64_t nb = (px + 31) / 32;
        const int64_t cost = (nb * sh.ks + (sh.s > 1 ? nb + kFsExchangeFixed : 0)) * wpc;
        if (best_cost < 0 || cost < best_cost) {
            best_cost = cost;
            best.shape = sh;
            best.pixels = (int)px;
            best.tile_rows = tr;
            best.wpc = wpc;
            best.width = width;
            best.window = width < p.pw;
            best.groups = ((int64_t)p.m + px - 1) / px;
            best.lds = lds;
        }
    }
    return best;
}

// LDS of the K-split kernel: every widened word of the region, or the
// reduction buffer (three partial copies of every 32x32 block), which
// reuses it; then the dot bounds of the workgroup's filters.
size_t mfma_ks_lds(const lce::MfmaParams &p, int mbw, int nblk, int tile_rows) {
    const size_t a = (size_t)p.cwe * tile_rows * p.pw * 16;
    const size_t red = (size_t)mbw * nblk * 3 * 16 * 64 * 4;
    return std::max(a, red) + (size_t)nblk * 32 * 4;
}

// The matrix-core launch parameters of a validated descriptor, all but the
// schedule's: x is the packed input, or (qf) the float32 input, 32 floats
// per packed word.  Fails with EUNSUPPORTED past the 2 GiB reach of the
// buffer loads; launches nothing.
lce_status mfma_params(const lce_bconv2d_desc &d, const Geometry &g, const void *x, bool qf,
                       const void *w_fp4, const float *multiplier, const float *bias,
                       const float *thresholds, const int32_t *flip, void *out,
                       lce::MfmaParams *pp) {
    lce::MfmaParams &p = *pp;
    p = lce::MfmaParams{};
    p.x = reinterpret_cast<const uint32_t *>(x);
    p.wexp = reinterpret_cast<const lce::u32x4 *>(w_fp4);
    p.mult = d.out_type == LCE_OUT_FLOAT32 ? multiplier : nullptr;
    p.bias = d.out_type == LCE_OUT_FLOAT32 ? bias : nullptr;
    p.thr = thresholds;
    p.flip = d.out_type == LCE_OUT_BITPACKED ? reinterpret_cast<const uint32_t *>(flip) : nullptr;
    p.out = out;
    int cc, cwe;
    p.n = d.n; p.h = d.h; p.w = d.w; p.cw = packed_words(d.c_in);
    mfma_chunk(p.cw, &cc, &cwe);
    p.cwe = cwe;
    p.oh = g.oh; p.ow = g.ow; p.cout = d.c_out; p.coutp = (d.c_out + 31) / 32 * 32;
    // the packed copy follows the widened filters in the same buffer
    p.wpk = reinterpret_cast<const uint32_t *>(p.wexp + (int64_t)d.kh * d.kw * cwe * p.coutp);
    p.cwo = packed_words(d.c_out);
    p.kh = d.kh; p.kw = d.kw; p.sh = d.stride_h; p.sw = d.stride_w; p.pt = g.pt; p.pl = g.pl;
    p.ph = (g.oh - 1) * d.stride_h + d.kh;
    p.pw = (g.ow - 1) * d.stride_w + d.kw;
    p.lo = d.clamp_min; p.hi = d.clamp_max;
    p.m = d.n * g.oh * g.ow;
    p.pad_zero = d.pad_value == LCE_PAD_ZERO ? 1 : 0;
    p.region_vec = !qf && p.cw % 4 == 0 && aligned(x, 16) ? 4 : 1;
    p.div_ohw = lce::make_fastdiv((uint32_t)(g.oh * g.ow));
    p.div_ow = lce::make_fastdiv((uint32_t)g.ow);
    p.div_ph = lce::make_fastdiv((uint32_t)p.ph);
    p.div_pw = lce::make_fastdiv((uint32_t)p.pw);

    p.div_cwh = lce::make_fastdiv((uint32_t)(p.cwe / 2));
    p.div_kw = lce::make_fastdiv((uint32_t)p.kw);
    p.div_groups = lce::make_fastdiv((uint32_t)(p.region_vec == 4 ? p.cw / 4 : p.cwe));
    // the filter-stationary and K-split kernels read the input and the
    // filters as buffers, with 32-bit byte offsets and offsets at or past
    // 2^31 standing for padding: each must stay below 2 GiB
    {
        const int64_t x_bytes = (int64_t)d.n * d.h * d.w * p.cw * (qf ? 128 : 4);
        const int64_t w_bytes = (int64_t)d.kh * d.kw * cwe * p.coutp * 16;
        if (x_bytes >= (int64_t(1) << 31) || w_bytes >= (int64_t(1) << 31))
            return fail(LCE_EUNSUPPORTED,
                        "the matrix-core path takes inputs and widened filters below 2 GiB "
                        "(input %lld bytes, widened filters %lld bytes)",
                        (long long)x_bytes, (long long)w_bytes);
    }
    return ok();
}

// Plans the filter-stationary schedule of a layer and launches it (qf: the
// input is float32, binarized while staged); false, with nothing launched,
// when no instance fits.
bool launch_fs_plan(lce::MfmaParams &p, const lce_bconv2d_desc &d, int64_t cus, int blocks32,
                    int64_t ksteps, bool qf, hipStream_t stream) {
    const FsPlan fp = plan_mfma_fs(p, cus, blocks32, (int)ksteps);
    if (!fp.shape.ks) return false;
    p.tile_rows = fp.tile_rows;
    p.fs_pixels = fp.pixels;
    p.fs_thr_off = (int32_t)(mfma_fs_thr_offset(fp.shape) / 4);
    if (fp.window) {        // the region: tile_rows x width from each share's first column
        p.pw = fp.width;
        p.div_pw = lce::make_fastdiv((uint32_t)fp.width);
    }
    p.div_plane = lce::make_fastdiv((uint32_t)(fp.tile_rows * p.pw));
    fill_step_table(p, d, fp.tile_rows * p.pw, (int)ksteps);
    size_t lds = fp.lds;
    // claim more than 1/(wpc+1) of a CU's LDS when the grid fits the
    // CUs, so that no CU holds more than wpc workgroups while another
    // holds fewer (tuning key mfma_fs_pad = -1 turns this off)
    const int64_t wgs = fp.groups * ((blocks32 + 4 / fp.shape.s - 1) / (4 / fp.shape.s));
    const int wpc = fp.wpc;
    if (tuning(LCE_TUNE_MFMA_FS_PAD) >= 0 && wgs <= cus * wpc &&
        lds * (wpc + 1) <= (size_t)device_max_lds())
        lds = std::max(lds, (size_t)device_max_lds() / (wpc + 1) + 1024);
    const dim3 grid((unsigned)fp.groups,
                    (unsigned)((blocks32 + 4 / fp.shape.s - 1) / (4 / fp.shape.s)));
    const bool pk = d.c_in == 32 * p.cwe && tuning(LCE_TUNE_MFMA_PACKED) >= 0;
    if (fp.window)
        lce::launch_mfma_fs_window(p, fp.shape.ks, fp.shape.s, pk, qf, d.out_type, grid, lds,
                                   stream);
    else
        lce::launch_mfma_fs(p, fp.shape.ks, fp.shape.s, pk, qf, d.out_type, grid, lds, stream);
    return true;
}

// The K-split plan of a layer: the tile of 32*MBW pixels x 32*NBLK filters
// is the largest (at most eight 32x32 blocks) whose grid still gives every
// CU 1.5 workgroups, among those whose LDS fits, else the one with the most
// workgroups; mbw == 0: none fits.
struct KsPlan {
    int mbw = 0, nblk = 0, tile_rows = 0;
    int64_t wgs = 0;
};

KsPlan plan_mfma_ks(const lce::MfmaParams &p, int64_t cus, int blocks32) {
    const int nmax = blocks32 >= 4 ? 4 : blocks32 >= 2 ? 2 : 1;
    static const int kTiles[][2] = {{4, 2}, {2, 4}, {2, 2}, {4, 1}, {1, 4},
                                    {2, 1}, {1, 2}, {1, 1}};
    KsPlan best;
    const int env_mb = tuning(LCE_TUNE_MFMA_TILE_M), env_nb = tuning(LCE_TUNE_MFMA_TILE_N);
    for (const auto &o : kTiles) {
        if (o[1] > nmax) continue;
        if (env_mb && o[0] != env_mb) continue;
        if (env_nb && o[1] != env_nb) continue;
        const int tr = mfma_tile_rows(p, 32 * o[0]);
        if (mfma_ks_lds(p, o[0], o[1], tr) > (size_t)device_max_lds()) continue;
        const int64_t wgs = ((int64_t)p.m + 32 * o[0] - 1) / (32 * o[0]) *
                            ((blocks32 + o[1] - 1) / o[1]);
        if (2 * wgs >= 3 * cus) return KsPlan{o[0], o[1], tr, wgs};
        if (wgs > best.wgs) best = KsPlan{o[0], o[1], tr, wgs};
    }
    return best;
}

// Launches the K-split plan `kp` (qf: the input is float32, binarized while
// staged); false, with nothing launched, when no tile fits.
bool launch_ks_plan(lce::MfmaParams &p, const lce_bconv2d_desc &d, const KsPlan &kp, int blocks32,
                    bool qf, hipStream_t stream) {
    if (!kp.mbw) return false;
    p.tile_rows = kp.tile_rows;
    p.div_plane = lce::make_fastdiv((uint32_t)(kp.tile_rows * p.pw));
    const size_t lds = mfma_ks_lds(p, kp.mbw, kp.nblk, kp.tile_rows);
    const dim3 grid((unsigned)(((int64_t)p.m + 32 * kp.mbw - 1) / (32 * kp.mbw)),
                    (unsigned)((blocks32 + kp.nblk - 1) / kp.nblk));
    p.div_ks_gx = lce::make_fastdiv(grid.x);
    lce::launch_mfma_ksplit(p, d.out_type, kp.nblk, kp.mbw, qf, grid, lds, stream);
    return true;
}

}  // namespace

extern "C" {

int32_t lce_packed_words(int32_t channels) {
    if (channels < 0) return -1;
    return packed_words(channels);
}

lce_status lce_bconv2d_out_shape(const lce_bconv2d_desc *desc, int32_t *oh, int32_t *ow) {
    if (!oh || !ow) return fail(LCE_EINVAL, "oh/ow output pointer is NULL");
    Geometry g;
    lce_status st = validate_desc(desc, &g);
    if (st != LCE_OK && st != LCE_EUNSUPPORTED) return st;
    *oh = g.oh;
    *ow = g.ow;
    return ok();
}

lce_status lce_bitpack(const float *x, int32_t *out, int64_t rows, int32_t channels,
                       hipStream_t stream) {
    if (rows < 0) return fail(LCE_EINVAL, "rows %lld < 0", (long long)rows);
    if (channels < 1) return fail(LCE_EINVAL, "channels %d < 1", channels);
    if (rows == 0) return ok();   // empty tensors may have null pointers
    if (!x || !out) return fail(LCE_EINVAL, "x/out is NULL");
    if (!aligned(x, 4) || !aligned(out, 4)) return fail(LCE_EALIGN, "x/out not 4-byte aligned");
    if (rows > (INT64_MAX / 64) / channels) return fail(LCE_EINVAL, "tensor too large");
    const int cw = packed_words(channels);
    const int64_t nwords = rows * cw;
    if (channels % 32 == 0 && aligned(x, 16)) {
        const int64_t chunks = (nwords + 7) / 8;
        const int64_t per_block = (lce::kBitpackThreads / 64) * lce::kBitpackUnroll;
        int64_t blocks = (chunks + per_block - 1) / per_block;
        if (blocks > 256 * 16) blocks = 256 * 16;
        hipLaunchKernelGGL(lce::bitpack32_kernel, dim3((unsigned)blocks),
                           dim3(lce::kBitpackThreads), 0, stream,
                           reinterpret_cast<const float4 *>(x), reinterpret_cast<uint32_t *>(out),
                           nwords);
    } else {
        int64_t blocks = (nwords + lce::kBitpackThreads - 1) / lce::kBitpackThreads;
        if (blocks > 256 * 32) blocks = 256 * 32;
        hipLaunchKernelGGL(lce::bitpack_generic_kernel, dim3((unsigned)blocks),
                           dim3(lce::kBitpackThreads), 0, stream, x,
                           reinterpret_cast<uint32_t *>(out), rows, (int)channels, cw);
    }
    return check_launch("lce_bitpack launch");
}

lce_status lce_bconv2d(const lce_bconv2d_desc *desc, const int32_t *x_packed,
                       const int32_t *w_packed, const float *multiplier, const float *bias,
                       const float *thresholds, const int32_t *flip,
                       const int32_t *pad_correction, void *out, hipStream_t stream) {
    Geometry g;
    lce_status st = validate_desc(desc, &g);
    if (st != LCE_OK) return st;
    const lce_bconv2d_desc &d = *desc;
    const bool padz = zero_padded(d, g);
    if (!x_packed || !w_packed || !out) return fail(LCE_EINVAL, "x_packed/w_packed/out is NULL");
    if (d.out_type == LCE_OUT_BITPACKED && !thresholds)
        return fail(LCE_EINVAL, "bitpacked output needs thresholds");
    if (padz && !pad_correction)
        return fail(LCE_EINVAL,
                    "zero padding on a padded geometry needs the pad_correction table");
    if (!aligned(x_packed, 4) || !aligned(w_packed, 4) || !aligned(out, 4) ||
        (multiplier && !aligned(multiplier, 4)) || (bias && !aligned(bias, 4)) ||
        (thresholds && !aligned(thresholds, 4)) || (flip && !aligned(flip, 4)) ||
        (pad_correction && !aligned(pad_correction, 4)))
        return fail(LCE_EALIGN, "tensor pointers must be 4-byte aligned");

    BconvParams p = bconv_params(d, g, w_packed, multiplier, bias, thresholds, flip, out);
    p.x = reinterpret_cast<const uint32_t *>(x_packed);
    p.padc = padz ? pad_correction : nullptr;
    p.slab = p.kwords < lce::kSlabWords ? p.kwords : lce::kSlabWords;
    p.rs = lce::row_stride(p.slab);

    const int filters = d.out_type == LCE_OUT_BITPACKED ? p.cwo * 32 : p.cout;
    if (has_static(p.cw, p.kh, p.kw) && input_fits_buffer(p)) {
        choose_schedule(p, filters);
    } else {
        p.nb = 1; p.ks = 1; p.fwg = lce::kWaves * lce::kRN; p.ksplit = p.kwords;
    }
    p.div_fwg = lce::make_fastdiv((uint32_t)p.fwg);
    dim3 grid((unsigned)((p.m + lce::kPix - 1) / lce::kPix),
              (unsigned)((filters + p.fwg - 1) / p.fwg));
    const int vec = aligned(x_packed, 16) ? 4 : aligned(x_packed, 8) ? 2 : 1;
    switch (d.out_type) {
        case LCE_OUT_FLOAT32: dispatch<lce::OUT_FLOAT>(p, grid, stream, vec, padz); break;
        case LCE_OUT_BITPACKED: dispatch<lce::OUT_BITS>(p, grid, stream, vec, padz); break;
        default: dispatch<lce::OUT_INT>(p, grid, stream, vec, padz); break;
    }
    return check_launch("lce_bconv2d launch");
}

// The quantize-fused kernel's schedule.  Every filter group binarizes its
// band again, so a second workgroup on a compute unit doubles that work:
// the smallest filter group (most groups, least GEMM per workgroup) whose
// grid still has at most one workgroup per compute unit; with more pixel
// blocks than compute units, one group of all filters (up to 128).
void choose_quant_schedule(BconvParams &p, int filters) {
    const long pix_blocks = (p.m + lce::kPix - 1) / lce::kPix;
    const long cus = device_simds() / 4;
    static const int kOptions[][2] = {{4, 1}, {2, 1}, {1, 1}, {1, 2}, {1, 4}};
    int nb = std::min(lce::kMaxNB, (filters + 31) / 32), ks = 1;
    for (const auto &o : kOptions) {
        if (o[1] > 1 && p.kwords < 4 * o[1]) continue;
        const long fwg = (lce::kWaves / o[1]) * o[0] * lce::kRN;
        if (pix_blocks * ((filters + fwg - 1) / fwg) <= cus) { nb = o[0]; ks = o[1]; }
    }
    if (const int t = tuning(LCE_TUNE_XOR_KS)) ks = t;
    if (const int t = tuning(LCE_TUNE_XOR_NB)) nb = t;
    if (ks != 1 && ks != 2 && ks != 4) ks = 1;
    if (ks > 1) nb = 1;
    nb = std::max(1, std::min(nb, lce::kMaxNB));
    p.ks = ks;
    p.nb = nb;
    p.fwg = (lce::kWaves / ks) * nb * lce::kRN;
    p.ksplit = ((p.kwords + ks - 1) / ks + 3) / 4 * 4;
}

lce_status lce_quantize_bconv2d(const lce_bconv2d_desc *desc, const float *x,
                                const int32_t *w_packed, const float *multiplier,
                                const float *bias, const float *thresholds,
                                const int32_t *flip, void *out, hipStream_t stream) {
    Geometry g;
    lce_status st = validate_desc(desc, &g);
    if (st != LCE_OK) return st;
    const lce_bconv2d_desc &d = *desc;
    // shapes the fused kernel does not cover: nothing is launched
    if (const char *why = quant_unsupported(d, g))
        return fail(LCE_EUNSUPPORTED, "%s; run lce_bitpack, then lce_bconv2d", why);
    if (!x || !w_packed || !out) return fail(LCE_EINVAL, "x/w_packed/out is NULL");
    if (d.out_type == LCE_OUT_BITPACKED && !thresholds)
        return fail(LCE_EINVAL, "bitpacked output needs thresholds");
    if (!aligned(x, 16))
        return fail(LCE_EALIGN, "x must be 16-byte aligned (it is read in 16-byte units)");
    if (!aligned(w_packed, 4) || !aligned(out, 4) || (multiplier && !aligned(multiplier, 4)) ||
        (bias && !aligned(bias, 4)) || (thresholds && !aligned(thresholds, 4)) ||
        (flip && !aligned(flip, 4)))
        return fail(LCE_EALIGN, "tensor pointers must be 4-byte aligned");

    BconvParams p = bconv_params(d, g, w_packed, multiplier, bias, thresholds, flip, out);
    p.xf = x;
    const int filters = d.out_type == LCE_OUT_BITPACKED ? p.cwo * 32 : p.cout;
    choose_quant_schedule(p, filters);
    p.div_fwg = lce::make_fastdiv((uint32_t)p.fwg);

    // Dynamic LDS: the im2col rows (later the K-split partial sums), then the
    // packed band.
    const int64_t rows = quant_band_rows(p);
    const int64_t band_words = rows * d.w * p.cw;
    const int64_t row_area = (int64_t)lce::kPix * lce::row_stride(p.kwords);
    const int64_t red_area = (int64_t)lce::kWaves * lce::kRN * lce::kPix;
    const int64_t first_area = (std::max(row_area, red_area) + 3) / 4 * 4;
    const int64_t lds = (first_area + (band_words + 3) / 4 * 4) * 4;
    const int64_t lds_static = (int64_t)lce::kMaxFiltersWG * 4;
    if (lds + lds_static > device_max_lds())
        return fail(LCE_EUNSUPPORTED,
                    "the input band of %lld rows needs %lld bytes of LDS (limit %d); run "
                    "lce_bitpack, then lce_bconv2d", (long long)rows,
                    (long long)(lds + lds_static), device_max_lds());
    p.band_rows = (int32_t)rows;
    p.band_pack = (int32_t)first_area;
    dim3 grid((unsigned)((p.m + lce::kPix - 1) / lce::kPix),
              (unsigned)((filters + p.fwg - 1) / p.fwg));
    lce::launch_bconv2d_quant(p, d.out_type, grid, (size_t)lds, stream);
    return check_launch("lce_quantize_bconv2d launch");
}

lce_status lce_bconv2d_pad_correction_size(const lce_bconv2d_desc *desc, int64_t *elements) {
    if (!elements) return fail(LCE_EINVAL, "elements output pointer is NULL");
    Geometry g;
    lce_status st = validate_desc(desc, &g);
    if (st != LCE_OK) return st;
    *elements = table_elements(*desc);
    return ok();
}

lce_status lce_bconv2d_pad_correction(const lce_bconv2d_desc *desc, const int32_t *w_packed,
                                      int32_t *pad_correction, hipStream_t stream) {
    Geometry g;
    lce_status st = validate_desc(desc, &g);
    if (st != LCE_OK) return st;
    const lce_bconv2d_desc &d = *desc;
    if (!w_packed || !pad_correction) return fail(LCE_EINVAL, "w_packed/pad_correction is NULL");
    if (!aligned(w_packed, 4) || !aligned(pad_correction, 4))
        return fail(LCE_EALIGN, "tensor pointers must be 4-byte aligned");
    const int64_t table = table_elements(d);
    if (table > INT32_MAX)
        return fail(LCE_EINVAL, "correction table of %lld elements exceeds 2^31",
                    (long long)table);
    const unsigned blocks = (unsigned)((d.c_out + 255) / 256);
    hipLaunchKernelGGL(lce::pad_table_kernel, dim3(blocks), dim3(256), 0, stream,
                       reinterpret_cast<const uint32_t *>(w_packed), pad_correction, d.c_out,
                       d.kh, d.kw, packed_words(d.c_in), d.c_in);
    return check_launch("lce_bconv2d_pad_correction launch");
}

// Converter-side fold of a float output transform followed by the next
// layer's binarization into a threshold and a direction per channel.  For an
// integer c, fmaf((float)c, m, b) < 0 exactly when c*m + b < 0 (c*m + b is a
// multiple of 2^-149, so it neither rounds to zero nor changes sign), and
// that is evaluated exactly in fp64 for |c| <= 2^24.  It is monotone in c:
// m > 0 gives "c < T" and m < 0 gives "not (c < T)" for the T found by
// bisection over the reachable clamped range; m == 0 gives the constant
// b < 0.
lce_status lce_fold_thresholds(const float *multiplier, const float *bias, int32_t c_out,
                               int32_t k, int32_t clamp_min, int32_t clamp_max,
                               float *thresholds, int32_t *flip) {
    if (!thresholds || !flip) return fail(LCE_EINVAL, "thresholds/flip is NULL");
    if (c_out < 1) return fail(LCE_EINVAL, "c_out %d < 1", c_out);
    if (k < 1 || k > (1 << 24)) return fail(LCE_EINVAL, "k %d outside [1, 2^24]", k);
    if (clamp_min > clamp_max)
        return fail(LCE_EINVAL, "clamp_min %d > clamp_max %d", clamp_min, clamp_max);
    for (int co = 0; co < c_out; ++co) {
        const float m = multiplier ? multiplier[co] : 1.0f;
        const float b = bias ? bias[co] : 0.0f;
        if (!std::isfinite(m) || !std::isfinite(b))
            return fail(LCE_EINVAL, "channel %d: multiplier %g / bias %g not finite", co,
                        (double)m, (double)b);
    }
    // reachable clamped accumulators: c = min(max(dot, lo), hi), |dot| <= k
    const int64_t cmin = std::min<int64_t>(std::max<int64_t>(-(int64_t)k, clamp_min), clamp_max);
    const int64_t cmax = std::min<int64_t>(std::max<int64_t>((int64_t)k, clamp_min), clamp_max);
    const float kInf = INFINITY;
    std::memset(flip, 0, sizeof(int32_t) * (size_t)packed_words(c_out));
    for (int co = 0; co < c_out; ++co) {
        const double m = multiplier ? (double)multiplier[co] : 1.0;
        const double b = bias ? (double)bias[co] : 0.0;
        auto neg = [&](int64_t c) { return (double)c * m + b < 0.0; };
        float thr;
        bool inv = false;
        if (m == 0.0) {
            thr = b < 0.0 ? kInf : -kInf;
        } else {
            // `lo_c` keeps the sign of cmin's side, `hi_c` the other one
            const bool at_min = neg(cmin), at_max = neg(cmax);
            if (at_min == at_max) {
                thr = at_min ? kInf : -kInf;
            } else {
                int64_t lo_c = cmin, hi_c = cmax;
                while (hi_c - lo_c > 1) {
                    const int64_t mid = lo_c + (hi_c - lo_c) / 2;
                    (neg(mid) == at_min ? lo_c : hi_c) = mid;
                }
                // hi_c is the first c whose sign differs from cmin's
                thr = (float)hi_c;
                inv = m < 0.0;   // negative for c >= hi_c: the inverse of c < hi_c
            }
        }
        thresholds[co] = thr;
        if (inv) flip[co / 32] |= (int32_t)(1u << (co % 32));
    }
    return ok();
}

lce_status lce_bmaxpool2d_out_shape(const lce_bmaxpool2d_desc *desc, int32_t *oh, int32_t *ow) {
    if (!oh || !ow) return fail(LCE_EINVAL, "oh/ow output pointer is NULL");
    Geometry g;
    lce_status st = validate_pool(desc, &g);
    if (st != LCE_OK) return st;
    *oh = g.oh;
    *ow = g.ow;
    return ok();
}

lce_status lce_bmaxpool2d(const lce_bmaxpool2d_desc *desc, const int32_t *x_packed,
                          int32_t *out, hipStream_t stream) {
    Geometry g;
    lce_status st = validate_pool(desc, &g);
    if (st != LCE_OK) return st;
    if (!x_packed || !out) return fail(LCE_EINVAL, "x_packed/out is NULL");
    if (!aligned(x_packed, 4) || !aligned(out, 4))
        return fail(LCE_EALIGN, "tensor pointers must be 4-byte aligned");
    const lce_bmaxpool2d_desc &d = *desc;
    lce::PoolParams p{};
    p.x = reinterpret_cast<const uint32_t *>(x_packed);
    p.out = reinterpret_cast<uint32_t *>(out);
    p.h = d.h; p.w = d.w; p.cw = packed_words(d.channels);
    p.oh = g.oh; p.ow = g.ow;
    p.kh = d.kh; p.kw = d.kw; p.sh = d.stride_h; p.sw = d.stride_w; p.pt = g.pt; p.pl = g.pl;
    const int vec = (p.cw % 4 == 0 && aligned(x_packed, 16) && aligned(out, 16)) ? 4
                    : (p.cw % 2 == 0 && aligned(x_packed, 8) && aligned(out, 8)) ? 2 : 1;
    const int64_t pixels = (int64_t)d.n * g.oh * g.ow;
    p.units = pixels * (p.cw / vec);
    p.div_cwv = lce::make_fastdiv((uint32_t)(p.cw / vec));
    p.div_ow = lce::make_fastdiv((uint32_t)g.ow);
    p.div_oh = lce::make_fastdiv((uint32_t)g.oh);
    if (vec == 4)
        launch_pool<4>(p, stream);
    else if (vec == 2)
        launch_pool<2>(p, stream);
    else
        launch_pool<1>(p, stream);
    return check_launch("lce_bmaxpool2d launch");
}

lce_status lce_dequantize(const int32_t *x_packed, float *out, int64_t rows, int32_t channels,
                          hipStream_t stream) {
    if (rows < 0) return fail(LCE_EINVAL, "rows %lld < 0", (long long)rows);
    if (channels < 1) return fail(LCE_EINVAL, "channels %d < 1", channels);
    if (rows == 0) return ok();   // empty tensors may have null pointers
    if (!x_packed || !out) return fail(LCE_EINVAL, "x_packed/out is NULL");
    if (!aligned(x_packed, 4) || !aligned(out, 4))
        return fail(LCE_EALIGN, "x_packed/out not 4-byte aligned");
    if (rows > (INT64_MAX / 64) / channels) return fail(LCE_EINVAL, "tensor too large");
    const int64_t count = rows * channels;
    if (channels % 32 == 0 && aligned(out, 16)) {
        const int64_t n4 = count / 4;
        int64_t blocks = (n4 + lce::kPoolThreads - 1) / lce::kPoolThreads;
        if (blocks > 256 * 16) blocks = 256 * 16;
        hipLaunchKernelGGL(lce::dequantize32_kernel, dim3((unsigned)blocks),
                           dim3(lce::kPoolThreads), 0, stream,
                           reinterpret_cast<const uint32_t *>(x_packed),
                           reinterpret_cast<float4 *>(out), n4);
    } else {
        int64_t blocks = (count + lce::kPoolThreads - 1) / lce::kPoolThreads;
        if (blocks > 256 * 16) blocks = 256 * 16;
        hipLaunchKernelGGL(lce::dequantize_generic_kernel, dim3((unsigned)blocks),
                           dim3(lce::kPoolThreads), 0, stream,
                           reinterpret_cast<const uint32_t *>(x_packed), out, count, channels,
                           packed_words(channels));
    }
    return check_launch("lce_dequantize launch");
}

lce_status lce_bconv2d_mfma_weights_size(const lce_bconv2d_desc *desc, int64_t *bytes) {
    if (!bytes) return fail(LCE_EINVAL, "bytes output pointer is NULL");
    Geometry g;
    lce_status st = validate_desc(desc, &g);
    if (st != LCE_OK) return st;
    *bytes = mfma_weight_bytes(*desc);
    return ok();
}

lce_status lce_bconv2d_mfma_weights(const lce_bconv2d_desc *desc, const int32_t *w_packed,
                                    void *w_fp4, hipStream_t stream) {
    Geometry g;
    lce_status st = validate_desc(desc, &g);
    if (st != LCE_OK) return st;
    const lce_bconv2d_desc &d = *desc;
    if (!w_packed || !w_fp4) return fail(LCE_EINVAL, "w_packed/w_fp4 is NULL");
    if (!aligned(w_packed, 4) || !aligned(w_fp4, 16))
        return fail(LCE_EALIGN, "w_packed must be 4-byte and w_fp4 16-byte aligned");
    int cc, cwe;
    const int cw = packed_words(d.c_in);
    mfma_chunk(cw, &cc, &cwe);
    const int coutp = (d.c_out + 31) / 32 * 32;
    const int taps = d.kh * d.kw;
    const int64_t total = (int64_t)taps * cwe * coutp;
    int64_t blocks = (total + 255) / 256;
    if (blocks > 256 * 16) blocks = 256 * 16;
    hipLaunchKernelGGL(lce::mfma_expand_weights_kernel, dim3((unsigned)blocks), dim3(256), 0,
                       stream, reinterpret_cast<const uint32_t *>(w_packed),
                       reinterpret_cast<lce::u32x4 *>(w_fp4),
                       reinterpret_cast<uint32_t *>(reinterpret_cast<lce::u32x4 *>(w_fp4) + total),
                       d.c_out, coutp, taps, cw, cwe, d.c_in);
    return check_launch("lce_bconv2d_mfma_weights launch");
}

lce_status lce_bconv2d_mfma(const lce_bconv2d_desc *desc, const int32_t *x_packed,
                            const void *w_fp4, const float *multiplier, const float *bias,
                            const float *thresholds, const int32_t *flip, void *out,
                            hipStream_t stream) {
    Geometry g;
    lce_status st = validate_desc(desc, &g);
    if (st != LCE_OK) return st;
    const lce_bconv2d_desc &d = *desc;
    if (!x_packed || !w_fp4 || !out) return fail(LCE_EINVAL, "x_packed/w_fp4/out is NULL");
    if (d.out_type == LCE_OUT_BITPACKED && !thresholds)
        return fail(LCE_EINVAL, "bitpacked output needs thresholds");
    if (!aligned(x_packed, 4) || !aligned(w_fp4, 16) || !aligned(out, 4) ||
        (multiplier && !aligned(multiplier, 4)) || (bias && !aligned(bias, 4)) ||
        (thresholds && !aligned(thresholds, 4)) || (flip && !aligned(flip, 4)))
        return fail(LCE_EALIGN, "tensor pointers must be 4-byte aligned (w_fp4 16-byte)");
    if ((int64_t)d.n * g.oh * g.ow > INT32_MAX - lce::kMfmaPixMax)
        return fail(LCE_EINVAL, "too many output pixels for the matrix-core path");
    const int64_t k = (int64_t)d.kh * d.kw * d.c_in;
    if (k >= (1 << 24))
        return fail(LCE_EUNSUPPORTED,
                    "K = %lld: the matrix-core path keeps dots exact in fp32 only below 2^24",
                    (long long)k);

    lce::MfmaParams p;
    st = mfma_params(d, g, x_packed, false, w_fp4, multiplier, bias, thresholds, flip, out, &p);
    if (st != LCE_OK) return st;
    int cc, cwe;
    mfma_chunk(p.cw, &cc, &cwe);
    const int64_t cus = device_simds() / 4;
    const int blocks32 = p.coutp / 32;
    const int nmax = blocks32 >= 4 ? 4 : blocks32 >= 2 ? 2 : 1;

    // K-split schedule (all four waves on one tile, K divided among them),
    // for long K: it widens the whole input region up front and ends with a
    // reduction, which pay off from about 5 K steps per wave on (measured
    // on the batch-1 sweep layers with 25 and 27 K steps, which no
    // filter-stationary instance covers within 1/8 padding: 3.7-5.7 us
    // against 7.4-10.2 us on the pixel split, whose K stages run one after
    // another behind barriers).  The tile is 32*MBW pixels x 32*NBLK
    // filters: the largest (at most eight 32x32 blocks) whose grid still
    // gives every CU 1.5 workgroups, among those whose LDS fits.  The
    // mfma_schedule tuning key forces either schedule (the K-split one where
    // its LDS fits).
    const int64_t ksteps = (int64_t)d.kh * d.kw * (p.cwe / 2);
    // 0 auto, 1 filter-stationary, 2 K split, 3 pixel split
    const int sched = tuning(LCE_TUNE_MFMA_SCHEDULE);
    const int ks_env = sched == 2 ? 1 : sched == 3 ? 0 : -1;

    // Filter-stationary schedule: the default wherever an instance fits, up
    // to 36 K steps.  Longer K runs on the K-split schedule below unless an
    // instance is forced (tuning keys mfma_fs_ks and mfma_fs_s): with S = 4
    // waves per filter block every filter group re-widens the same input
    // region and the partial sums add LDS traffic, measured slower than the
    // K split on the 7x7x512 layer.  The mfma_schedule key forces one of the
    // others.
    const bool fs_forced = tuning(LCE_TUNE_MFMA_FS_KS) && tuning(LCE_TUNE_MFMA_FS_S);
    if (ks_env < 0 &&
        (ksteps <= 36 || (fs_forced && ksteps <= 72))) {
        if (launch_fs_plan(p, d, cus, blocks32, ksteps, false, stream))
            return check_launch("lce_bconv2d_mfma launch");
    }

    if (ks_env == 1 || (ks_env != 0 && ksteps >= 20)) {
        if (launch_ks_plan(p, d, plan_mfma_ks(p, cus, blocks32), blocks32, false, stream))
            return check_launch("lce_bconv2d_mfma launch");
    }

    // Pixel-split schedule: MB pixel blocks of 32 per wave (128*MB pixels
    // per workgroup) and NBLK filter blocks of 32, one channel chunk widened
    // at a time (any region width that fits one chunk).  The largest tiles
    // reuse each operand read from LDS most; they are kept while the grid
    // still covers every CU.
    static const int kSplits[][2] = {{2, 4}, {1, 4}, {2, 2}, {1, 2}, {2, 1}, {1, 1}};
    int mb = 1, nblk = 1;
    int64_t best_wgs = -1;
    for (const auto &o : kSplits) {
        if (o[1] > nmax) continue;
        const int64_t wgs = ((int64_t)p.m + 128 * o[0] - 1) / (128 * o[0]) *
                            ((blocks32 + o[1] - 1) / o[1]);
        if (wgs >= cus) { mb = o[0]; nblk = o[1]; break; }
        if (wgs > best_wgs) { best_wgs = wgs; mb = o[0]; nblk = o[1]; }
    }
    if (const int t = tuning(LCE_TUNE_MFMA_TILE_N)) nblk = t;
    if (const int t = tuning(LCE_TUNE_MFMA_TILE_M)) mb = t;
    if (nblk != 1 && nblk != 2 && nblk != 4) nblk = 4;
    if (mb != 1 && mb != 2) mb = 2;
    const int bm = 128 * mb;
    p.tile_rows = mfma_tile_rows(p, bm);
    p.div_plane = lce::make_fastdiv((uint32_t)(p.tile_rows * p.pw));
    const int64_t pix_groups = ((int64_t)p.m + bm - 1) / bm;
    // dynamic LDS: the widened A chunk, the packed input region (with the
    // 256-word slack of its last DMA instruction), one byte per region row;
    // the four B stages are static (4 x CC x 32*NBLK x 16 bytes)
    const size_t region_words = (size_t)p.tile_rows * p.pw * p.cw;
    const size_t lds = (size_t)cc * p.tile_rows * p.pw * 16 + (region_words + 256) * 4 +
                       ((size_t)p.tile_rows + 15) / 16 * 16;
    const size_t lds_static = (size_t)4 * cc * 32 * nblk * 16;
    if (lds + lds_static > (size_t)device_max_lds())
        return fail(LCE_EUNSUPPORTED,
                    "matrix-core tile of %zu bytes exceeds the %d bytes of LDS per workgroup "
                    "(padded width %d, %d rows)", lds + lds_static, device_max_lds(), p.pw,
                    p.tile_rows);
    if ((int64_t)p.tile_rows * p.pw * cc > INT32_MAX / 2)
        return fail(LCE_EUNSUPPORTED, "matrix-core tile too large");
    const dim3 grid((unsigned)pix_groups, (unsigned)((blocks32 + nblk - 1) / nblk));
    lce::launch_mfma_pixel(p, d.out_type, cc, nblk, mb, grid, lds, stream);
    return check_launch("lce_bconv2d_mfma launch");
}

lce_status lce_quantize_bconv2d_mfma(const lce_bconv2d_desc *desc, const float *x,
                                     const void *w_fp4, const float *multiplier,
                                     const float *bias, const float *thresholds,
                                     const int32_t *flip, void *out, hipStream_t stream) {
    Geometry g;
    lce_status st = validate_desc(desc, &g);
    if (st != LCE_OK) return st;
    const lce_bconv2d_desc &d = *desc;
    if (!x || !w_fp4 || !out) return fail(LCE_EINVAL, "x/w_fp4/out is NULL");
    if (d.out_type == LCE_OUT_BITPACKED && !thresholds)
        return fail(LCE_EINVAL, "bitpacked output needs thresholds");
    if (!aligned(x, 16) || !aligned(w_fp4, 16))
        return fail(LCE_EALIGN, "x and w_fp4 must be 16-byte aligned (16-byte loads)");
    if (!aligned(out, 4) || (multiplier && !aligned(multiplier, 4)) ||
        (bias && !aligned(bias, 4)) || (thresholds && !aligned(thresholds, 4)) ||
        (flip && !aligned(flip, 4)))
        return fail(LCE_EALIGN, "out and the per-channel arrays must be 4-byte aligned");
    if (d.c_in % 32 != 0)
        return fail(LCE_EUNSUPPORTED,
                    "c_in %d is not a multiple of 32; run lce_bitpack, then lce_bconv2d_mfma",
                    d.c_in);
    if ((int64_t)d.n * g.oh * g.ow > INT32_MAX - lce::kMfmaPixMax)
        return fail(LCE_EINVAL, "too many output pixels for the matrix-core path");
    const int64_t k = (int64_t)d.kh * d.kw * d.c_in;
    if (k >= (1 << 24))
        return fail(LCE_EUNSUPPORTED,
                    "K = %lld: the matrix-core path keeps dots exact in fp32 only below 2^24",
                    (long long)k);
    lce::MfmaParams p;
    st = mfma_params(d, g, x, true, w_fp4, multiplier, bias, thresholds, flip, out, &p);
    if (st != LCE_OK) return st;
    // the schedules that stage the region through registers, by the same
    // plans as lce_bconv2d_mfma's: filter-stationary where one of its
    // instances takes the shape, else the K split from 20 K steps (the pixel
    // split stages by LDS DMA and is not fused).  From 37 to 72 K steps the
    // filter-stationary schedule also comes first where the K split's grid
    // has fewer workgroups than CUs: each of those few workgroups stages a
    // large region, and a float region costs 32 times the packed bytes
    // (batch-1 7x7x512: 32 workgroups, 6.96 us, against 6.31 us on the
    // (18, 4) instance; at batch 64, 392 workgroups, the K split is faster,
    // 20.6 vs 22.2 us).  The mfma_schedule key restricts the choice to one
    // schedule (the filter-stationary one then up to 72 K steps).
    const int64_t ksteps = (int64_t)d.kh * d.kw * (p.cwe / 2);
    const int sched = tuning(LCE_TUNE_MFMA_SCHEDULE);   // 0 auto, 1 FS, 2 K split, 3 pixel
    const bool fs_k = (sched == 0 || sched == 1) && ksteps <= 72 && fs_any_takes(ksteps);
    const bool ks_k = (sched == 0 && ksteps >= 20) || sched == 2;
    if (fs_k || ks_k) {
        const int64_t cus = device_simds() / 4;
        const int blocks32 = p.coutp / 32;
        const KsPlan kp = ks_k ? plan_mfma_ks(p, cus, blocks32) : KsPlan{};
        const bool fs_first =
            fs_k && (ksteps <= 36 || sched == 1 || !kp.mbw || kp.wgs < cus);
        if ((fs_first && launch_fs_plan(p, d, cus, blocks32, ksteps, true, stream)) ||
            (ks_k && launch_ks_plan(p, d, kp, blocks32, true, stream)))
            return check_launch("lce_quantize_bconv2d_mfma launch");
    }
    return fail(LCE_EUNSUPPORTED,
                "neither the filter-stationary nor the K-split schedule takes this shape "
                "(%lld K steps%s); run lce_bitpack, then lce_bconv2d_mfma", (long long)ksteps,
                sched ? ", schedule restricted by the mfma_schedule tuning key" : "");
}

lce_status lce_set_tuning(int32_t key, int32_t value) {
    if (key < 0 || key >= LCE_TUNE_COUNT) return fail(LCE_EINVAL, "unknown tuning key %d", key);
    g_tuning[key].store(value, std::memory_order_relaxed);
    return ok();
}

int32_t lce_get_tuning(int32_t key) {
    if (key < 0 || key >= LCE_TUNE_COUNT) return 0;
    return g_tuning[key].load(std::memory_order_relaxed);
}

const char *lce_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
