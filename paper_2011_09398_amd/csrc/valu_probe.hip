// Throughput probe for the binary convolution's inner loop: the highest rate
// at which a gfx950 CU retires v_xor_b32 (one scalar operand) followed by
// v_bcnt_u32_b32 (popcount + accumulate), with no memory traffic.  This is
// the measured ceiling the convolution's VALU roofline fraction is quoted
// against, next to the 256 CU x 64 lane x 2.4 GHz spec figure.
//
// Each lane runs `iters` rounds of RN x KC independent xor/bcnt pairs; the
// empty asm statements keep the operands opaque so nothing is hoisted.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr int kRN = 8, kKC = 8;

__global__ __launch_bounds__(256) void xor_popcount_probe(const uint32_t *__restrict__ seed,
                                                          uint32_t *__restrict__ out,
                                                          int iters) {
    uint32_t a[kKC];
#pragma unroll
    for (int j = 0; j < kKC; ++j) a[j] = seed[(threadIdx.x + j) & 63] ^ blockIdx.x;
    uint32_t w[kRN][kKC];
#pragma unroll
    for (int f = 0; f < kRN; ++f)
#pragma unroll
        for (int j = 0; j < kKC; ++j) w[f][j] = seed[64 + f * kKC + j];   // uniform: SGPRs
    uint32_t acc[kRN];
#pragma unroll
    for (int f = 0; f < kRN; ++f) acc[f] = 0;
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int j = 0; j < kKC; ++j) {
            asm("" : "+v"(a[j]));
#pragma unroll
            for (int f = 0; f < kRN; ++f) {
                acc[f] = __builtin_popcount(a[j] ^ w[f][j]) + acc[f];
                asm("" : "+v"(acc[f]));
            }
        }
    }
    uint32_t s = 0;
#pragma unroll
    for (int f = 0; f < kRN; ++f) s += acc[f];
    out[blockIdx.x * 256 + threadIdx.x] = s;
}

}  // namespace

// Launches `blocks` x 256 threads; each thread retires iters*8*8 xor/bcnt
// pairs.  seed: >= 128 device words; out: >= blocks*256 device words.
extern "C" int lce_probe_xor_popcount(const uint32_t *seed, uint32_t *out, int blocks,
                                      int iters, hipStream_t stream) {
    if (!seed || !out || blocks < 1 || iters < 1) return 1;
    hipLaunchKernelGGL(xor_popcount_probe, dim3(blocks), dim3(256), 0, stream, seed, out, iters);
    return hipGetLastError() == hipSuccess ? 0 : 4;
}

// xor/bcnt pairs one call retires, for the host's rate computation.
extern "C" long long lce_probe_pairs(int blocks, int iters) {
    return (long long)blocks * 256 * iters * kRN * kKC;
}
