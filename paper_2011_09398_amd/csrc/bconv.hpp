// Bitpacked binary 2-D convolution (LceBConv2d, arXiv 2011.09398 Section 3.2)
// as one fused kernel: implicit im2col -> XOR/POPCOUNT GEMM -> output transform.
//
// Work decomposition (gfx950, wave64):
//   * a workgroup is 4 waves and owns 64 consecutive output pixels
//     m = (n, oy, ox); lane l of every wave computes pixel m0 + l;
//   * each wave owns RN consecutive filters (wave-uniform), so the packed
//     filter words are uniform across the wave and live in scalar registers
//     (s_load), feeding v_xor_b32 as its scalar operand;
//   * the 64 pixels' im2col rows (KH*KW*Cw words each) are staged in LDS,
//     padded taps written as 0 words (= +1.0, one-padding), so the hot loop
//     is only LDS reads plus v_xor_b32 / v_bcnt_u32_b32 (popcount+accumulate);
//   * the accumulator stays in VGPRs and the output transform is applied
//     before anything is written (clamp, then fma or threshold compare).
//
// The filter words of a wave are read in the same k order as the im2col row
// (OHWI filters: k = (ky*KW + kx)*Cw + cw), so the GEMM's k loop is one
// contiguous walk over both.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lce {

enum OutKind : int { OUT_FLOAT = 0, OUT_BITS = 1, OUT_INT = 2 };

constexpr int kPix = 64;      // output pixels per workgroup (one per lane)
constexpr int kWaves = 4;     // waves per workgroup
constexpr int kThreads = kPix * kWaves;
constexpr int kSlabWords = 160;   // max im2col words staged per row at once

struct BconvParams {
    const uint32_t *x;      // [N][H][W][Cw]
    const uint32_t *w;      // [Cout][KH][KW][Cw]
    const float *mult;      // [Cout] or null
    const float *bias;      // [Cout] or null
    const float *thr;       // [Cout] (bitpacked output)
    void *out;
    int32_t n, h, wd, cw;
    int32_t oh, ow, cout, cwo;
    int32_t kh, kw, sh, sw, pt, pl;
    int32_t kwords;         // KH*KW*Cw
    int32_t k;              // KH*KW*C_in, the number of +-1 products
    int32_t lo, hi;         // fused activation bounds
    int32_t m;              // N*OH*OW
    int32_t ohw;            // OH*OW
    int32_t slab;           // generic kernel: words staged per pass
    int32_t rs;             // generic kernel: LDS row stride (words)
};

// LDS row stride for a row of `words` words: a multiple of 4 (16-byte rows
// for ds_read_b128) with an odd number of 16-byte quads, so the rows of
// neighbouring lanes start in different bank groups.
__host__ __device__ constexpr int row_stride(int words) {
    return ((words + 3) / 4) % 2 == 1 ? (words + 3) / 4 * 4 : (words + 3) / 4 * 4 + 4;
}

template <int N>
__device__ __forceinline__ void lds_read(uint32_t (&a)[N], const uint32_t *p) {
    static_assert(N % 4 == 0, "chunk is a whole number of 16-byte reads");
#pragma unroll
    for (int i = 0; i < N; i += 4) {
        const uint4 v = *reinterpret_cast<const uint4 *>(p + i);
        a[i] = v.x; a[i + 1] = v.y; a[i + 2] = v.z; a[i + 3] = v.w;
    }
}

// acc += popcount(a XOR w) as one v_bcnt_u32_b32 (popcount plus accumulate).
// The empty asm pins the running sum to a register after every step, so the
// compiler cannot re-associate a chunk's popcounts into an add tree (which
// costs an extra v_add3 per two words).
__device__ __forceinline__ void bcnt_acc(uint32_t &acc, uint32_t x) {
    acc = __builtin_popcount(x) + acc;
    asm("" : "+v"(acc));
}

// acc[f] += sum_k popcount(a_k XOR w[f][k]) over `nwords` words starting at
// word 0 of `arow` (LDS) and of each filter row `wrow + f*kwords` (global,
// wave-uniform).  FULL: all RN filters exist; otherwise filters past `nvalid`
// re-read the last valid row (results unused) so no load leaves the tensor.
template <int RN, int KC, bool FULL>
__device__ __forceinline__ void xor_popcount(uint32_t (&acc)[RN], const uint32_t *arow,
                                             const uint32_t *__restrict__ wrow, int kwords,
                                             int nwords, int nvalid) {
    int k = 0;
    for (; k + KC <= nwords; k += KC) {
        uint32_t a[KC];
        lds_read<KC>(a, arow + k);
#pragma unroll
        for (int j = 0; j < KC; ++j) {
#pragma unroll
            for (int f = 0; f < RN; ++f) {
                const int fo = FULL ? f : min(f, nvalid - 1);
                bcnt_acc(acc[f], a[j] ^ wrow[(size_t)fo * kwords + k + j]);
            }
        }
    }
    for (; k < nwords; ++k) {
        const uint32_t a0 = arow[k];
#pragma unroll
        for (int f = 0; f < RN; ++f) {
            const int fo = FULL ? f : min(f, nvalid - 1);
            bcnt_acc(acc[f], a0 ^ wrow[(size_t)fo * kwords + k]);
        }
    }
}

template <int VEC> struct VecOf;
template <> struct VecOf<4> {
    using type = uint4;
    __device__ static uint4 zero() { return make_uint4(0, 0, 0, 0); }
};
template <> struct VecOf<2> {
    using type = uint2;
    __device__ static uint2 zero() { return make_uint2(0, 0); }
};
template <> struct VecOf<1> {
    using type = uint32_t;
    __device__ static uint32_t zero() { return 0u; }
};

// Output transform of one lane's RN accumulators (Section 3.2: the fused
// activation and the per-channel multiplier/bias, or the threshold compare,
// applied to the accumulator before it is written).
template <int RN, int OUT>
__device__ __forceinline__ void epilogue(const BconvParams &p, const uint32_t (&acc)[RN],
                                         int m, int co0) {
    const int nvalid = min(RN, p.cout - co0);   // may be <= 0 for pad-bit waves
    if constexpr (OUT == OUT_BITS) {
        uint32_t bits = 0;
#pragma unroll
        for (int f = 0; f < RN; ++f) {
            if (f < nvalid) {
                const int dot = p.k - 2 * (int)acc[f];
                const int c = min(max(dot, p.lo), p.hi);
                if ((double)c < (double)p.thr[co0 + f]) bits |= 1u << f;
            }
        }
        uint8_t *o = reinterpret_cast<uint8_t *>(p.out) + (size_t)m * p.cwo * 4 + co0 / 8;
        if constexpr (RN == 8) {
            *o = (uint8_t)bits;
        } else if constexpr (RN == 16) {
            *reinterpret_cast<uint16_t *>(o) = (uint16_t)bits;
        } else {
            static_assert(RN == 32, "bitpacked output needs 8, 16 or 32 filters per wave");
            *reinterpret_cast<uint32_t *>(o) = bits;
        }
    } else if constexpr (OUT == OUT_FLOAT) {
        float *o = reinterpret_cast<float *>(p.out) + (size_t)m * p.cout + co0;
#pragma unroll
        for (int f = 0; f < RN; ++f) {
            if (f < nvalid) {
                const int dot = p.k - 2 * (int)acc[f];
                const int c = min(max(dot, p.lo), p.hi);
                const float mu = p.mult ? p.mult[co0 + f] : 1.0f;
                const float bi = p.bias ? p.bias[co0 + f] : 0.0f;
                o[f] = __builtin_fmaf((float)c, mu, bi);
            }
        }
    } else {
        int32_t *o = reinterpret_cast<int32_t *>(p.out) + (size_t)m * p.cout + co0;
#pragma unroll
        for (int f = 0; f < RN; ++f) {
            if (f < nvalid) {
                const int dot = p.k - 2 * (int)acc[f];
                o[f] = min(max(dot, p.lo), p.hi);
            }
        }
    }
}

// Shape-specialized kernel: Cw, KH, KW known at compile time, so the whole
// im2col row fits one LDS slab and the filter-row offsets are immediates.
// VEC = words per global load when staging (needs x aligned to 4*VEC bytes).
template <int CW, int KH, int KW, int RN, int KC, int VEC, int OUT>
__global__ __launch_bounds__(kThreads) void bconv2d_static_kernel(BconvParams p) {
    constexpr int kTaps = KH * KW;
    constexpr int kWords = kTaps * CW;
    constexpr int kRS = row_stride(kWords);
    __shared__ __attribute__((aligned(16))) uint32_t lds[kPix * kRS];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int m = blockIdx.x * kPix + lane;
    const bool px_ok = m < p.m;

    // ---- stage the im2col rows: wave w copies taps w, w+4, ... of every pixel.
    // All global loads are issued before any LDS store; a padded tap loads
    // from the image's first pixel (always in bounds) and is replaced by 0.
    {
        int img = 0, oy = 0, ox = 0;
        if (px_ok) {
            img = m / p.ohw;
            const int r = m - img * p.ohw;
            oy = r / p.ow;
            ox = r - oy * p.ow;
        }
        const int iy0 = oy * p.sh - p.pt;
        const int ix0 = ox * p.sw - p.pl;
        const uint32_t *ximg = p.x + (size_t)img * p.h * p.wd * CW;
        constexpr int kIters = (kTaps + kWaves - 1) / kWaves;
        constexpr int kVecs = CW / VEC;
        using Vec = typename VecOf<VEC>::type;
        Vec v[kIters][kVecs];
        bool in[kIters];
#pragma unroll
        for (int i = 0; i < kIters; ++i) {
            const int t = min(wave + i * kWaves, kTaps - 1);
            const int ky = t / KW, kx = t - (t / KW) * KW;
            const int iy = iy0 + ky, ix = ix0 + kx;
            in[i] = px_ok && (unsigned)iy < (unsigned)p.h && (unsigned)ix < (unsigned)p.wd;
            const size_t off = in[i] ? ((size_t)iy * p.wd + ix) * CW : 0;
            const Vec *src = reinterpret_cast<const Vec *>(ximg + off);
#pragma unroll
            for (int c = 0; c < kVecs; ++c) v[i][c] = src[c];
        }
        uint32_t *row = lds + lane * kRS;
#pragma unroll
        for (int i = 0; i < kIters; ++i) {
            const int t = wave + i * kWaves;
            if (t < kTaps) {
                Vec *dst = reinterpret_cast<Vec *>(row + t * CW);
#pragma unroll
                for (int c = 0; c < kVecs; ++c) dst[c] = in[i] ? v[i][c] : VecOf<VEC>::zero();
            }
        }
    }
    __syncthreads();

    const int co0 = (blockIdx.y * kWaves + wave) * RN;
    uint32_t acc[RN];
#pragma unroll
    for (int f = 0; f < RN; ++f) acc[f] = 0;
    if (co0 < p.cout) {
        const uint32_t *arow = lds + lane * kRS;
        const uint32_t *wrow = p.w + (size_t)co0 * kWords;
        if (co0 + RN <= p.cout)
            xor_popcount<RN, KC, true>(acc, arow, wrow, kWords, kWords, RN);
        else
            xor_popcount<RN, KC, false>(acc, arow, wrow, kWords, kWords, p.cout - co0);
    }
    if (!px_ok) return;
    if (OUT == OUT_BITS ? co0 >= p.cwo * 32 : co0 >= p.cout) return;
    epilogue<RN, OUT>(p, acc, m, co0);
}

// Generic kernel: any Cw/KH/KW.  The im2col row is staged in slabs of
// p.slab words (k range [k0, k0+slab)), one word per copy.
template <int RN, int KC, int OUT>
__global__ __launch_bounds__(kThreads) void bconv2d_generic_kernel(BconvParams p) {
    extern __shared__ __attribute__((aligned(16))) uint32_t lds_dyn[];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int m = blockIdx.x * kPix + lane;
    const bool px_ok = m < p.m;
    int img = 0, oy = 0, ox = 0;
    if (px_ok) {
        img = m / p.ohw;
        const int r = m - img * p.ohw;
        oy = r / p.ow;
        ox = r - oy * p.ow;
    }
    const int iy0 = oy * p.sh - p.pt;
    const int ix0 = ox * p.sw - p.pl;
    const uint32_t *ximg = p.x + (size_t)img * p.h * p.wd * p.cw;
    uint32_t *row = lds_dyn + lane * p.rs;

    const int co0 = (blockIdx.y * kWaves + wave) * RN;
    uint32_t acc[RN];
#pragma unroll
    for (int f = 0; f < RN; ++f) acc[f] = 0;

    for (int k0 = 0; k0 < p.kwords; k0 += p.slab) {
        const int nw = min(p.slab, p.kwords - k0);
        if (k0 > 0) __syncthreads();   // every wave is done with the previous slab
        for (int kk = wave; kk < nw; kk += kWaves) {
            const int kidx = k0 + kk;
            const int tap = kidx / p.cw;
            const int c = kidx - tap * p.cw;
            const int ky = tap / p.kw, kx = tap - (tap / p.kw) * p.kw;
            const int iy = iy0 + ky, ix = ix0 + kx;
            const bool in = px_ok && (unsigned)iy < (unsigned)p.h && (unsigned)ix < (unsigned)p.wd;
            const size_t off = in ? ((size_t)iy * p.wd + ix) * p.cw + c : 0;
            row[kk] = in ? ximg[off] : 0u;
        }
        __syncthreads();
        if (co0 < p.cout) {
            const uint32_t *wrow = p.w + (size_t)co0 * p.kwords + k0;
            if (co0 + RN <= p.cout)
                xor_popcount<RN, KC, true>(acc, row, wrow, p.kwords, nw, RN);
            else
                xor_popcount<RN, KC, false>(acc, row, wrow, p.kwords, nw, p.cout - co0);
        }
    }
    if (!px_ok) return;
    if (OUT == OUT_BITS ? co0 >= p.cwo * 32 : co0 >= p.cout) return;
    epilogue<RN, OUT>(p, acc, m, co0);
}

}  // namespace lce
