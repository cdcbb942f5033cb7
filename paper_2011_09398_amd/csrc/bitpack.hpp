// Sign binarization + bitpacking (LceQuantize, arXiv 2011.09398 Section 3.2).
//
// Bit c%32 of word c/32 of a row is 1 iff x[row][c] < 0.0f (a 1 bit stands
// for -1.0, a 0 bit for +1.0); bits past the channel count are 0.
//
// The work is HBM-bound (4 bytes read per bit written), so the kernels are
// shaped for coalesced loads: in the fast path a wave reads 1 KiB of
// contiguous floats per instruction (one float4 per lane), each lane turns
// its four signs into a nibble, and three DPP row shifts OR the nibbles of
// eight neighbouring lanes into the 32-bit word they make up.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dpp.hpp"

namespace lce {

constexpr int kBitpackThreads = 256;
constexpr int kBitpackUnroll = 4;   // 1 KiB chunks in flight per wave

// Fast path: channels % 32 == 0 and x 16-byte aligned, so the tensor is a
// flat sequence of 32-float groups, each packing into one word.
// A chunk is 64 float4 = 256 floats = 8 words.
__global__ __launch_bounds__(kBitpackThreads) void bitpack32_kernel(
    const float4 *__restrict__ x, uint32_t *__restrict__ out, int64_t nwords) {
    const int lane = threadIdx.x & 63;
    const int64_t nvec = nwords * 8;            // float4 count
    const int64_t nchunks = (nwords + 7) / 8;
    const int64_t wave = ((int64_t)blockIdx.x * kBitpackThreads + threadIdx.x) >> 6;
    const int64_t nwaves = ((int64_t)gridDim.x * kBitpackThreads) >> 6;
    const int shift = 4 * (lane & 7);
    for (int64_t c0 = wave * kBitpackUnroll; c0 < nchunks; c0 += nwaves * kBitpackUnroll) {
        float4 v[kBitpackUnroll];
#pragma unroll
        for (int u = 0; u < kBitpackUnroll; ++u) {
            const int64_t idx = (c0 + u) * 64 + lane;
            v[u] = idx < nvec ? x[idx] : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int u = 0; u < kBitpackUnroll; ++u) {
            uint32_t nib = (uint32_t)(v[u].x < 0.0f) | ((uint32_t)(v[u].y < 0.0f) << 1) |
                           ((uint32_t)(v[u].z < 0.0f) << 2) | ((uint32_t)(v[u].w < 0.0f) << 3);
            uint32_t s = nib << shift;
            s |= row_shr<1>(s);
            s |= row_shr<2>(s);
            s |= row_shr<4>(s);
            // Lane 8g+7 now holds the OR over lanes 8g..8g+7: word g of the chunk.
            const int64_t word = (c0 + u) * 8 + (lane >> 3);
            if ((lane & 7) == 7 && word < nwords) out[word] = s;
        }
    }
}

// General path: any channel count and 4-byte alignment; one thread per word.
__global__ __launch_bounds__(kBitpackThreads) void bitpack_generic_kernel(
    const float *__restrict__ x, uint32_t *__restrict__ out, int64_t rows, int channels,
    int cw) {
    const int64_t total = rows * (int64_t)cw;
    const int64_t stride = (int64_t)gridDim.x * kBitpackThreads;
    for (int64_t i = (int64_t)blockIdx.x * kBitpackThreads + threadIdx.x; i < total; i += stride) {
        const int64_t r = i / cw;
        const int j = (int)(i - r * cw);
        const float *src = x + r * channels + (int64_t)j * 32;
        const int nb = min(32, channels - j * 32);
        uint32_t word = 0;
        for (int b = 0; b < nb; ++b) word |= (uint32_t)(src[b] < 0.0f) << b;
        out[i] = word;
    }
}

}  // namespace lce
