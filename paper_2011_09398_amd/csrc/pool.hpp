// The operators on either side of the binary convolution that act on
// bitpacked tensors (arXiv 2011.09398 Section 3.2):
//
//   LceBMaxPool2d  max pooling of +-1 activations, computed on the packed
//                  bits.  max(sign(x)) = sign(max(x)), and the maximum of
//                  +-1 values is -1 only when every value is -1, i.e. when
//                  every bit is 1: the pooled word is the bitwise AND of the
//                  window's words.  Locations outside the image take no part
//                  (TensorFlow max pooling), which the AND identity (all
//                  ones) gives for free.  Pad bits stay 0 (0 AND anything).
//   LceDequantize  packed bits back to +-1.0 floats: bit 1 -> -1.0f,
//                  bit 0 -> +1.0f, built directly as the IEEE pattern
//                  0x3F800000 | bit << 31.
//
// Both are memory-bound: one thread per output word vector (pooling) or per
// output float4 (dequantize), consecutive threads on consecutive addresses,
// grid-stride loops over a grid of at most a few workgroups per CU.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bconv.hpp"   // FastDiv

namespace lce {

constexpr int kPoolThreads = 256;

struct PoolParams {
    const uint32_t *x;      // [N][H][W][Cw]
    uint32_t *out;          // [N][OH][OW][Cw]
    int32_t h, w, cw;
    int32_t oh, ow;
    int32_t kh, kw, sh, sw, pt, pl;
    int64_t units;          // output vectors: N*OH*OW*(Cw/VEC), below 2^31
    FastDiv div_cwv;        // unit -> pixel (Cw/VEC vectors per pixel)
    FastDiv div_ow;         // pixel -> output row
    FastDiv div_oh;         // output row -> image
};

template <int VEC> struct WordVec;
template <> struct WordVec<4> {
    using type = uint4;
    __device__ static uint4 ones() { return make_uint4(~0u, ~0u, ~0u, ~0u); }
    __device__ static uint4 and_(uint4 a, uint4 b) {
        return make_uint4(a.x & b.x, a.y & b.y, a.z & b.z, a.w & b.w);
    }
};
template <> struct WordVec<2> {
    using type = uint2;
    __device__ static uint2 ones() { return make_uint2(~0u, ~0u); }
    __device__ static uint2 and_(uint2 a, uint2 b) { return make_uint2(a.x & b.x, a.y & b.y); }
};
template <> struct WordVec<1> {
    using type = uint32_t;
    __device__ static uint32_t ones() { return ~0u; }
    __device__ static uint32_t and_(uint32_t a, uint32_t b) { return a & b; }
};

// Binary max pooling: one thread per VEC consecutive words of one output
// pixel.  KH, KW > 0: window size known at compile time; 0: read from p.
// Input and output word counts stay below 2^31 (checked on the host).
template <int VEC, int KH, int KW>
__global__ __launch_bounds__(kPoolThreads) void bmaxpool_kernel(PoolParams p) {
    using V = WordVec<VEC>;
    using T = typename V::type;
    const int kh = KH > 0 ? KH : p.kh, kw = KW > 0 ? KW : p.kw;
    const uint32_t stride = gridDim.x * kPoolThreads;
    const uint32_t cwv = p.div_cwv.d;
    for (uint32_t u = blockIdx.x * kPoolThreads + threadIdx.x; u < (uint32_t)p.units;
         u += stride) {
        const uint32_t pix = fast_div(u, p.div_cwv);
        const uint32_t q = u - pix * cwv;
        const uint32_t row = fast_div(pix, p.div_ow);
        const int ox = (int)(pix - row * (uint32_t)p.ow);
        const uint32_t img = fast_div(row, p.div_oh);
        const int oy = (int)(row - img * (uint32_t)p.oh);
        const int iy0 = oy * p.sh - p.pt, ix0 = ox * p.sw - p.pl;
        const T *base = reinterpret_cast<const T *>(p.x + img * (uint32_t)(p.h * p.w * p.cw)) + q;
        // Straight-line window (constant trip counts unroll fully at -O3): a
        // tap outside the image loads a clamped in-image location and is
        // replaced by the AND identity, so every load is issued at once.
        T acc = V::ones();
        for (int ky = 0; ky < kh; ++ky) {
            const int iy = iy0 + ky;
            const bool row_in = (unsigned)iy < (unsigned)p.h;
            const uint32_t cy = (uint32_t)min(max(iy, 0), p.h - 1);
            for (int kx = 0; kx < kw; ++kx) {
                const int ix = ix0 + kx;
                const bool in = row_in && (unsigned)ix < (unsigned)p.w;
                const uint32_t cx = (uint32_t)min(max(ix, 0), p.w - 1);
                const T v = base[(cy * (uint32_t)p.w + cx) * cwv];
                acc = V::and_(acc, in ? v : V::ones());
            }
        }
        reinterpret_cast<T *>(p.out)[u] = acc;
    }
}

// Dequantize, channels a multiple of 32 (and out 16-byte aligned): output
// float4 j holds channels 4*(j % 8) .. +3 of word j / 8.
__global__ __launch_bounds__(kPoolThreads) void dequantize32_kernel(const uint32_t *__restrict__ x,
                                                                    float4 *__restrict__ out,
                                                                    int64_t n4) {
    const int64_t stride = (int64_t)gridDim.x * kPoolThreads;
    for (int64_t j = (int64_t)blockIdx.x * kPoolThreads + threadIdx.x; j < n4; j += stride) {
        const uint32_t nib = x[j >> 3] >> ((j & 7) * 4);
        float4 v;
        v.x = __uint_as_float(0x3F800000u | (nib & 1u) << 31);
        v.y = __uint_as_float(0x3F800000u | (nib >> 1 & 1u) << 31);
        v.z = __uint_as_float(0x3F800000u | (nib >> 2 & 1u) << 31);
        v.w = __uint_as_float(0x3F800000u | (nib >> 3 & 1u) << 31);
        out[j] = v;
    }
}

// Dequantize, any channel count: one output float per thread.
__global__ __launch_bounds__(kPoolThreads) void dequantize_generic_kernel(
    const uint32_t *__restrict__ x, float *__restrict__ out, int64_t count, int channels,
    int cw) {
    const int64_t stride = (int64_t)gridDim.x * kPoolThreads;
    for (int64_t i = (int64_t)blockIdx.x * kPoolThreads + threadIdx.x; i < count; i += stride) {
        const int64_t r = i / channels;
        const int c = (int)(i - r * channels);
        const uint32_t bit = (x[r * cw + (c >> 5)] >> (c & 31)) & 1u;
        out[i] = __uint_as_float(0x3F800000u | bit << 31);
    }
}

}  // namespace lce
