// LceQuantize fused into the binary convolution that consumes it (arXiv
// 2011.09398 Section 3.2: a float activation is sign-binarized and
// bitpacked, then convolved), as one launch with no communication between
// workgroups.  The input arrives as float32 NHWC with a channel count that
// is a multiple of 32.
//
// A workgroup owns 64 consecutive output pixels (one per lane) and a group
// of filters, as in the XOR/POPCOUNT static kernel.  Their windows read a
// band of input rows that is contiguous in memory: global rows n*H + y from
// the first pixel's first in-image row to the last pixel's last one (a band
// may run across an image boundary).  The workgroup
//   1. loads the band's floats with coalesced 16-byte loads (a wave reads
//      1 KiB per instruction, up to 16 of them in flight per wave);
//   2. binarizes them in registers: four sign tests make a nibble and three
//      DPP row shifts OR eight nibbles into a packed word (bit c%32 of word
//      c/32 is x < 0.0f, the test of the bitpack kernel), written to a
//      packed band in LDS;
//   3. builds each pixel's im2col row from the packed band, padded taps as
//      0 words (one padding);
//   4. runs the XOR/POPCOUNT GEMM and the output transform of the static
//      kernel (compute_and_store).
// Each filter group binarizes its band again: the launch trades that
// redundant work (VALU) for the separate bitpack launch and its round trip
// through memory, which is what pays at small batches.  The host sizes the
// LDS for the tallest band of the launch (band_rows) and rejects shapes
// whose band does not fit.
#pragma once

#include "bconv.hpp"
#include "dpp.hpp"

namespace lce {

// Global input rows [first, last] read by the windows of output pixels
// [m_a, m_b] (wave-uniform).
__device__ __forceinline__ void band_rows(const BconvParams &p, int m_a, int m_b, int kh,
                                          int &first, int &last) {
    const uint32_t ohw = p.div_ohw.d;
    const uint32_t img_a = fast_div((uint32_t)m_a, p.div_ohw);
    const uint32_t oy_a = fast_div((uint32_t)m_a - img_a * ohw, p.div_ow);
    const uint32_t img_b = fast_div((uint32_t)m_b, p.div_ohw);
    const uint32_t oy_b = fast_div((uint32_t)m_b - img_b * ohw, p.div_ow);
    first = (int)img_a * p.h + max(0, (int)oy_a * p.sh - p.pt);
    last = (int)img_b * p.h + min(p.h - 1, (int)oy_b * p.sh - p.pt + kh - 1);
}

// CW: packed words per pixel (C_in = 32*CW).  Dynamic LDS: words
// [0, p.band_pack) hold the im2col rows and the K-split partial sums, words
// [p.band_pack, ...) the packed band.
template <int CW, int KH, int KW, int OUT>
__global__ __launch_bounds__(kThreads) void bconv2d_quant_kernel(BconvParams p) {
    constexpr int kTaps = KH * KW;
    constexpr int kWords = kTaps * CW;
    constexpr int kRS = row_stride(kWords);
    constexpr int VEC = CW % 4 == 0 ? 4 : CW % 2 == 0 ? 2 : 1;
    using Vec = typename VecOf<VEC>::type;
    extern __shared__ __attribute__((aligned(16))) uint32_t dyn[];
    __shared__ __attribute__((aligned(16))) uint32_t bound[kMaxFiltersWG];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int m_a = blockIdx.x * kPix;
    const int m = m_a + lane;
    const bool px_ok = m < p.m;
    const int co_wg = blockIdx.y * p.fwg;

    int first, last;
    band_rows(p, m_a, min(m_a + kPix - 1, p.m - 1), KH, first, last);
    first = __builtin_amdgcn_readfirstlane(first);
    const int rows = min(__builtin_amdgcn_readfirstlane(last) - first + 1, p.band_rows);
    const int row_words = p.wd * CW;
    const int words = rows * row_words;              // packed band words
    const int vecs = words * 8;                      // float4 in the band

    // ---- 1-2. binarize the band into LDS.  Chunk u = 64 float4 (8 packed
    // words); wave w takes chunks w, w+4, ..., kU of them per round, every
    // load of a round issued before the first is used.  The loads are not
    // predicated (a conditional load makes the compiler wait for every load
    // before it): chunks past the band re-read its last float4, and are
    // skipped (uniform branch) when binarizing.  Lane 8g+7 of chunk u
    // assembles packed word 8u+g.
    load_bounds<OUT, false>(p, co_wg, p.fwg, bound);
    uint32_t *packed = dyn + p.band_pack;
    {
        constexpr int kU = 16;
        const float4 *src = reinterpret_cast<const float4 *>(p.xf) +
                            (size_t)first * (size_t)row_words * 8;
        const int chunks = (vecs + 63) / 64;
        const int shift = 4 * (lane & 7);
        for (int base = 0; base < chunks; base += kWaves * kU) {
            float4 f[kU];
#pragma unroll
            for (int i = 0; i < kU; ++i)
                f[i] = src[min((base + i * kWaves + wave) * 64 + lane, vecs - 1)];
#pragma unroll
            for (int i = 0; i < kU; ++i) {
                const int u = base + i * kWaves + wave;
                if (u < chunks) {
                    const uint32_t nib = (uint32_t)(f[i].x < 0.0f) |
                                         ((uint32_t)(f[i].y < 0.0f) << 1) |
                                         ((uint32_t)(f[i].z < 0.0f) << 2) |
                                         ((uint32_t)(f[i].w < 0.0f) << 3);
                    uint32_t w = nib << shift;
                    w |= row_shr<1>(w);
                    w |= row_shr<2>(w);
                    w |= row_shr<4>(w);
                    const int word = u * 8 + (lane >> 3);
                    if ((lane & 7) == 7 && word < words) packed[word] = w;
                }
            }
        }
    }
    __syncthreads();

    // ---- 3. im2col rows from the packed band (wave w copies taps w, w+4, ...).
    // An in-image tap of a valid pixel lies in band row img*H + y - first,
    // inside [0, rows).
    {
        int y0 = 0, x0 = 0, base = 0;
        if (px_ok) {
            const uint32_t img = fast_div((uint32_t)m, p.div_ohw);
            const uint32_t r = (uint32_t)m - img * p.div_ohw.d;
            const uint32_t oy = fast_div(r, p.div_ow);
            const uint32_t ox = r - oy * (uint32_t)p.ow;
            y0 = (int)oy * p.sh - p.pt;
            x0 = (int)ox * p.sw - p.pl;
            base = (int)img * p.h - first;
        }
        uint32_t *row = dyn + lane * kRS;
#pragma unroll
        for (int t = wave; t < kTaps; t += kWaves) {
            const int ky = t / KW, kx = t - (t / KW) * KW;
            const int y = y0 + ky, x = x0 + kx;
            const bool in = px_ok && (unsigned)y < (unsigned)p.h && (unsigned)x < (unsigned)p.wd;
            const Vec *src = reinterpret_cast<const Vec *>(
                packed + (in ? ((base + y) * p.wd + x) * CW : 0));
            Vec *dst = reinterpret_cast<Vec *>(row + t * CW);
#pragma unroll
            for (int c = 0; c < CW / VEC; ++c) dst[c] = in ? src[c] : VecOf<VEC>::zero();
        }
    }
    __syncthreads();
    compute_and_store<kRN, kKC, OUT, false>(p, dyn + lane * kRS, kWords, wave, lane, m, co_wg,
                                            bound, nullptr, PadWin16(), dyn);
}

}  // namespace lce
