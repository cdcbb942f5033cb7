// Bitpacked binary 2-D convolution (LceBConv2d, arXiv 2011.09398 Section 3.2)
// on the gfx950 matrix cores.
//
// The binary convolution is a dense contraction of +-1 values: dot =
// sum_k a_k * w_k.  Section 3.2 evaluates it with XOR + POPCOUNT because the
// paper's CPUs have no faster way to multiply +-1 values.  gfx950 has one:
// its MFMA multiplies 4-bit floats (e2m1), in which +1.0 and -1.0 (and 0.0)
// are exact, and accumulates in fp32, which is exact for every |dot| < 2^24.
// The MFMA therefore returns the same integer dot, at a dense rate (10.1
// PFLOP/s) eight times the VALU's xor+popcount rate.  The data stay
// bitpacked in memory; each 1-bit value is widened to a 4-bit +-1.0 only in
// LDS, right before the matrix cores read it.
//
// Instruction: v_mfma_scale_f32_32x32x64_f8f6f4 with both operands fp4 and
// unit scales (E8M0 127 = 2^0).  Lane l holds row (or column) l % 32 and one
// block of 32 consecutive k values, l / 32 choosing the block.  A dot product
// does not depend on the order of k, so a lane's block is simply one packed
// word (32 channels of one tap) widened to 16 bytes; the filter side is
// widened the same way once per filter tensor (mfma_expand_weights_kernel).
//
// Work decomposition: a workgroup (4 waves) owns 128*MB consecutive output
// pixels and 32*NBLK filters; each wave computes MB blocks of 32 pixels
// against all the workgroup's filters (MB x NBLK 32x32 accumulator blocks),
// so every B operand it reads from LDS feeds MB matrix products.
//   * A: the input region the 128 pixels read (rows of the batch stacked as
//     padded images, all padded columns) is widened once per channel chunk
//     of CC words into LDS; every tap of the im2col is then an address
//     offset into it, so a word is widened once, not once per tap.
//     Padding locations widen to +1.0 (one-padding, Section 3.2) or 0.0
//     (zero padding): zero padding costs nothing on this path.
//   * B: the widened filters of one tap and chunk (a stage), streamed into
//     LDS by DMA through four slots, three stages ahead of the one in use.
//   * Epilogue: the fp32 accumulator is the exact integer dot; the fused
//     activation clamp and the float transform or threshold compare follow
//     as on the XOR path.  Bitpacked output gathers each pixel's 32 filter
//     bits with one ballot per accumulator row pair.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <utility>

#include "bconv.hpp"   // FastDiv, OutKind, thr_to_padz-style bounds

namespace lce {

constexpr int kMfmaPixMax = 256;   // output pixels per workgroup (32 or 64 per wave)

// 16 bytes as a native vector (HIP's uint4 is a class, which keeps arrays of
// it out of registers)
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr int kMfmaThreads = 256;

// e2m1 codes: +1.0 = 0x2, -1.0 = 0xA.  Byte for two bits (lo, hi):
// code(lo) | code(hi) << 4, indexed by lo | hi << 1.
constexpr uint32_t kFp4PlusMinusLut = 0xAAA22A22u;
// Byte for two validity bits: 0xF for each valid half, 0x0 otherwise.
constexpr uint32_t kFp4ValidLut = 0xFFF00F00u;

struct MfmaParams {
    const uint32_t *x;      // [N][H][W][Cw] bitpacked activations
    const u32x4 *wexp;      // [KH*KW*CwE][CoutP] widened filters (16 bytes = 32 values)
    const float *mult;      // [Cout] or null (float output)
    const float *bias;      // [Cout] or null (float output)
    const float *thr;       // [Cout] (bitpacked output)
    const uint32_t *flip;   // [Cwo] or null (bitpacked output)
    void *out;
    int32_t n, h, w, cw, cwe;        // cwe: Cw rounded up to a multiple of CC
    int32_t oh, ow, cout, coutp, cwo;
    int32_t kh, kw, sh, sw, pt, pl;
    int32_t ph, pw;                  // padded image: (OH-1)*sh + KH rows, (OW-1)*sw + KW cols
    int32_t lo, hi, m;
    int32_t tile_rows;               // stacked padded rows staged per workgroup
    int32_t pad_zero;                // 1: padded locations are 0.0
    int32_t region_vec;              // words per DMA lane when staging the region: 4 or 1
    FastDiv div_ohw, div_ow, div_ph, div_pw;
    FastDiv div_plane;               // tile_rows * pw: region locations
    FastDiv div_cwh, div_kw;         // cwe / 2 (word pairs per tap), kw
    FastDiv div_groups;              // region_vec-word groups per location
};

typedef int mfma_v8i __attribute__((ext_vector_type(8)));
typedef float mfma_v16f __attribute__((ext_vector_type(16)));


// One packed byte -> four bytes holding its 2-bit groups (bits 2i, 2i+1 of
// x land in bits 0-1 of byte i).
__device__ __forceinline__ uint32_t spread_pairs(uint32_t x) {
    uint32_t t = ((x << 12) | x) & 0x000F000Fu;
    return ((t << 6) | t) & 0x03030303u;
}

// Packed word -> 32 e2m1 codes (16 bytes), channel c in nibble c of the
// result (little-endian): the lookup `lut` maps each 2-bit group to a byte
// (kFp4PlusMinusLut for +-1.0, 0 for all 0.0).
__device__ __forceinline__ u32x4 widen_word(uint32_t w, uint32_t lut) {
    u32x4 o;
    o.x = __builtin_amdgcn_perm(lut, lut, spread_pairs(w & 0xFFu));
    o.y = __builtin_amdgcn_perm(lut, lut, spread_pairs((w >> 8) & 0xFFu));
    o.z = __builtin_amdgcn_perm(lut, lut, spread_pairs((w >> 16) & 0xFFu));
    o.w = __builtin_amdgcn_perm(lut, lut, spread_pairs(w >> 24));
    return o;
}

__device__ __forceinline__ mfma_v16f mfma_fp4(u32x4 a, u32x4 b, mfma_v16f c) {
    const mfma_v8i av = {(int)a.x, (int)a.y, (int)a.z, (int)a.w, 0, 0, 0, 0};
    const mfma_v8i bv = {(int)b.x, (int)b.y, (int)b.z, (int)b.w, 0, 0, 0, 0};
    // operand formats 4 = e2m1; scales 127 = 2^0
    return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av, bv, c, 4, 4, 0, 127, 0, 127);
}

// Threshold as a bound on the unclamped dot, as a float: bit = clamp(dot) <
// thr becomes dot < T with T = ceil(thr) inside (lo, hi] (|T| <= 2^24 there
// is not needed: T only meets exact integer dots below 2^24), +infinity when
// ceil(thr) > hi (always), -infinity when ceil(thr) <= lo or thr is NaN
// (never).  The fp32 accumulator holds the dot exactly, so the compare is
// one v_cmp_lt_f32 whose lane mask is the output bits.
__device__ inline float thr_to_dot_bound_f(float thr, int lo, int hi) {
    const double t = (double)thr;
    if (t != t) return -INFINITY;
    const double tc = ceil(t);
    if (tc <= (double)lo) return -INFINITY;
    if (tc > (double)hi) return INFINITY;
    return (float)tc;
}

// Bitpacked output of one 32x32 accumulator block.  Value v of the block is
// pixel (v/4)*8 + half*4 + v%4 and filter lane % 32, so one ballot of
// "value < T" over the wave gives the 32 filter bits of two pixels (lanes
// 0-31 and 32-63); v_writelane drops each 32-bit half into the lane of its
// pixel.  fmask (wave-uniform) flips chosen filters.  Lane l < 32 returns
// the word of pixel l.
//
// The SGPR a v_writelane reads may have just been written by a VALU
// instruction (the compare itself, when there is no flip mask).  CDNA3/4
// require two wait states between the two that the hardware does not
// insert, and the compiler's hazard recognizer does not look inside inline
// asm, so each v_writelane carries its own s_nop 1.
template <int V>
__device__ __forceinline__ void block_bits_step(const mfma_v16f &val, float T, uint64_t fmask,
                                                uint32_t &word) {
    constexpr int r0 = (V >> 2) * 8 + (V & 3);
    const uint64_t mask = __ballot(val[V] < T) ^ fmask;
    asm("s_nop 1\n\tv_writelane_b32 %0, %1, %2" : "+v"(word) : "s"((uint32_t)mask), "i"(r0));
    asm("s_nop 1\n\tv_writelane_b32 %0, %1, %2"
        : "+v"(word) : "s"((uint32_t)(mask >> 32)), "i"(r0 + 4));
}
template <int... V>
__device__ __forceinline__ uint32_t block_bits_impl(const mfma_v16f &val, float T,
                                                    uint64_t fmask,
                                                    std::integer_sequence<int, V...>) {
    uint32_t word = 0;
    (block_bits_step<V>(val, T, fmask, word), ...);
    return word;
}
__device__ __forceinline__ uint32_t block_bits(const mfma_v16f &val, float T, uint64_t fmask) {
    return block_bits_impl(val, T, fmask, std::make_integer_sequence<int, 16>{});
}

// Flip mask of a block of 32 filters for both lane halves, wave-uniform:
// flip word `fw` restricted to the filters below C_out (co_ok per lane).
__device__ __forceinline__ uint64_t block_flip(const uint32_t *flip, int word_index, bool co_ok) {
    if (!flip) return 0;
    const uint32_t fw = __builtin_amdgcn_readfirstlane(flip[word_index]);
    const uint32_t fv = (uint32_t)__ballot(co_ok ? 1u : 0u) & fw;
    return (uint64_t)fv | ((uint64_t)fv << 32);
}

// Stacked padded row of output pixel m's window origin, and its column.
__device__ __forceinline__ void mfma_pixel(const MfmaParams &p, int m, int &row, int &col) {
    const uint32_t img = fast_div((uint32_t)m, p.div_ohw);
    const uint32_t r = (uint32_t)m - img * p.div_ohw.d;
    const uint32_t oy = fast_div(r, p.div_ow);
    const uint32_t ox = r - oy * (uint32_t)p.ow;
    row = (int)img * p.ph + (int)oy * p.sh;
    col = (int)ox * p.sw;
}

// 16 zero bytes in device memory: the DMA source of every padding word.
__device__ __attribute__((aligned(16))) const uint32_t g_mfma_zero[4] = {0u, 0u, 0u, 0u};

typedef __attribute__((address_space(1))) void mfma_global_void;
typedef __attribute__((address_space(3))) void mfma_lds_void;

// s_waitcnt vmcnt(N) alone (expcnt and lgkmcnt fields at their maxima).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | 0x70 | 0xF00);
}

// s_waitcnt lgkmcnt(0) alone (vmcnt and expcnt fields at their maxima).
__device__ __forceinline__ void wait_lgkmcnt0() { __builtin_amdgcn_s_waitcnt(0xC07F); }

// Workgroup barrier for the pipelined loop: this wave's LDS accesses done
// (lgkmcnt), then s_barrier.  Unlike __syncthreads() it carries no memory
// fence, whose release semantics would make the compiler wait for every LDS
// DMA in flight; the DMA stages the loop needs are waited for explicitly
// (vmcnt) before it.  Without a fence nothing stops the compiler from
// moving an LDS read above the barrier, so the barrier returns an opaque
// zero, produced after it, that every read of barrier-protected LDS adds to
// its address.
__device__ __forceinline__ int lds_barrier() {
    int zero;
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier\n\tv_mov_b32 %0, 0"
                 : "=v"(zero) : : "memory");
    return zero;
}

template <int CC, int OUT, int NBLK, int MB>
__global__ __launch_bounds__(kMfmaThreads) void bconv2d_mfma_kernel(MfmaParams p) {
    constexpr int BN = 32 * NBLK;
    constexpr int BM = 32 * MB * 4;                                   // pixels per workgroup
    constexpr int kStage = CC * BN;                                   // u32x4 per B stage
    constexpr int kDmaPerStage = kStage / 64;                         // 1 KB instructions
    constexpr int kDmaPerWave = (kDmaPerStage + 3) / 4;
    // B stages: four separate arrays, so that the compiler can tell the
    // stage being read from the ones being written by DMA
    __shared__ __attribute__((aligned(16))) u32x4 bslot0[kStage];
    __shared__ __attribute__((aligned(16))) u32x4 bslot1[kStage];
    __shared__ __attribute__((aligned(16))) u32x4 bslot2[kStage];
    __shared__ __attribute__((aligned(16))) u32x4 bslot3[kStage];
    extern __shared__ __attribute__((aligned(16))) u32x4 smem[];
    const int tid = threadIdx.x;
    const int lane = tid & 63, half = lane >> 5, l32 = lane & 31;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int m0 = blockIdx.x * BM;
    const int n_base = blockIdx.y * BN;
    const int taps = p.kh * p.kw;
    const int chunks = p.cwe / CC;
    const int stages = chunks * taps;
    const int TR = p.tile_rows, PW = p.pw, plane = TR * PW;
    const int bits_words = plane * p.cw;                      // packed input region
    const int V = p.region_vec;
    u32x4 *atile = smem;                                      // [CC][TR][PW] e2m1
    // packed region, word-group major: [Cw/V][TR][PW][V], so that the lanes
    // widening one word of consecutive locations read consecutive addresses
    uint32_t *abits = reinterpret_cast<uint32_t *>(atile + CC * plane);
    uint8_t *rowok = reinterpret_cast<uint8_t *>(abits + bits_words + 256);  // [TR]

    int row0, col0;
    mfma_pixel(p, m0, row0, col0);
    // A rows of this lane: pixel blocks b = 0..MB-1 of the wave
    int a_base[MB];
#pragma unroll
    for (int b = 0; b < MB; ++b) {
        const int mp = min(m0 + (wave * MB + b) * 32 + l32, p.m - 1);
        int prow, pcol;
        mfma_pixel(p, mp, prow, pcol);
        a_base[b] = (half * TR + (prow - row0)) * PW + pcol;
    }

    // ---- the packed input region by LDS DMA: element q = g*plane + rc holds
    // words [g*V, g*V + V) of region location rc = r*PW + c; padding reads
    // the zero buffer.  Each lane moves one element (16 bytes when Cw is a
    // multiple of 4); the last instruction's extra lanes land in the 256-word
    // slack after the region.
    auto stage_region = [&](auto vec_c) __attribute__((always_inline)) {
        constexpr int V = decltype(vec_c)::value;
        for (int u = wave; u * 64 * V < bits_words; u += 4) {
            const int q = min(u * 64 + lane, bits_words / V - 1);
            const int g = (int)fast_div((uint32_t)q, p.div_plane);
            const int rc = q - g * plane;
            const int j = g * V;
            const int r = (int)fast_div((uint32_t)rc, p.div_pw);
            const int c = rc - r * PW;
            const int R = row0 + r;
            const int img = (int)fast_div((uint32_t)R, p.div_ph);
            const int yy = R - img * p.ph - p.pt, xx = c - p.pl;
            const bool inside = img < p.n && (unsigned)yy < (unsigned)p.h &&
                                (unsigned)xx < (unsigned)p.w;
            const uint32_t *src =
                inside ? p.x + (((size_t)img * p.h + yy) * p.w + xx) * p.cw + j : g_mfma_zero;
            if constexpr (V == 4)
                __builtin_amdgcn_global_load_lds((mfma_global_void *)src,
                                                 (mfma_lds_void *)(abits + u * 64 * V), 16, 0, 0);
            else
                __builtin_amdgcn_global_load_lds((mfma_global_void *)src,
                                                 (mfma_lds_void *)(abits + u * 64 * V), 4, 0, 0);
        }
    };
    if (p.region_vec == 4)
        stage_region(std::integral_constant<int, 4>{});
    else
        stage_region(std::integral_constant<int, 1>{});
    // rows of the region that are image rows (zero padding needs them)
    for (int r = tid; r < TR; r += kMfmaThreads) {
        const int R = row0 + r;
        const int img = (int)fast_div((uint32_t)R, p.div_ph);
        const int yy = R - img * p.ph - p.pt;
        rowok[r] = (uint8_t)(img < p.n && (unsigned)yy < (unsigned)p.h);
    }

    // ---- B stage s = (chunk s / taps, tap s % taps) by LDS DMA into `slot`:
    // words [c0, c0+CC) of the tap, filters [n_base, n_base + BN); DMA
    // instruction u moves elements e = 64u + lane, e = j*BN + f.  Stages past
    // the last re-read it (the loop below always issues the same number of
    // instructions, which keeps the vmcnt accounting exact).
    auto issue_b = [&](int s, u32x4 *slot) __attribute__((always_inline)) {
        s = min(s, stages - 1);
        const int c0 = (s / taps) * CC, t = s - (s / taps) * taps;
#pragma unroll
        for (int i = 0; i < kDmaPerWave; ++i) {
            const int u = wave + 4 * i;
            if (u < kDmaPerStage) {
                const int e = u * 64 + lane;
                const int j = e / BN, f = e - (e / BN) * BN;
                const int co = min(n_base + f, p.coutp - 1);
                const u32x4 *src = p.wexp + (size_t)(t * p.cwe + c0 + j) * p.coutp + co;
                __builtin_amdgcn_global_load_lds((mfma_global_void *)src,
                                                 (mfma_lds_void *)(slot + u * 64), 16, 0, 0);
            }
        }
    };
    issue_b(0, bslot0);
    issue_b(1, bslot1);
    issue_b(2, bslot2);

    // per-lane output-transform parameters of the NBLK filters this lane
    // stores (loaded now, used after the last stage)
    float ep_a[NBLK], ep_b[NBLK];
#pragma unroll
    for (int i = 0; i < NBLK; ++i) {
        const int co = min(n_base + 32 * i + l32, p.cout - 1);
        if constexpr (OUT == OUT_BITS) {
            ep_a[i] = p.thr[co];
            ep_b[i] = 0.0f;
        } else if constexpr (OUT == OUT_FLOAT) {
            ep_a[i] = p.mult ? p.mult[co] : 1.0f;
            ep_b[i] = p.bias ? p.bias[co] : 0.0f;
        } else {
            ep_a[i] = ep_b[i] = 0.0f;
        }
    }

    mfma_v16f acc[MB][NBLK];
#pragma unroll
    for (int b = 0; b < MB; ++b)
#pragma unroll
        for (int i = 0; i < NBLK; ++i)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[b][i][v] = 0.0f;

    // widen words [c0, c0+CC) of the region into the A tile (LDS -> LDS);
    // padding locations are 0 words, i.e. +1.0, unless zero padding asks 0.0
    // (with 16-byte elements a chunk is exactly one element: CC = 4 = V)
    auto widen_chunk = [&](int c0, int z) __attribute__((always_inline)) {
        for (int rc = tid; rc < plane; rc += kMfmaThreads) {
            uint32_t lut = kFp4PlusMinusLut;
            if (p.pad_zero) {
                const int r = (int)fast_div((uint32_t)rc, p.div_pw);
                const int xx = rc - r * PW - p.pl;
                if (!(rowok[r + z] && (unsigned)xx < (unsigned)p.w)) lut = 0u;
            }
            uint32_t bits[CC];
            if (CC == 4 && V == 4) {
                const u32x4 b4 = reinterpret_cast<const u32x4 *>(abits)[(c0 >> 2) * plane + rc + z];
#pragma unroll
                for (int j = 0; j < CC; ++j) bits[j] = b4[j];
            } else {
#pragma unroll
                for (int j = 0; j < CC; ++j)
                    bits[j] = c0 + j < p.cw ? abits[(c0 + j) * plane + rc + z] : 0u;
            }
#pragma unroll
            for (int j = 0; j < CC; ++j) atile[j * plane + rc] = widen_word(bits[j], lut);
        }
    };

    // Operands of one stage in registers, double-buffered: stage s reads its
    // A and B operands from LDS and then issues the matrix products of stage
    // s-1, whose operands arrived during the previous stage, so that the LDS
    // reads of one stage overlap the matrix products of the other.
    typedef u32x4 OpsA[CC / 2][MB];
    typedef u32x4 OpsB[CC / 2][NBLK];
    OpsA oa0, oa1;
    OpsB ob0, ob1;
    auto load_ops = [&](int t, const u32x4 *cur, int z, OpsA &oa, OpsB &ob)
                        __attribute__((always_inline)) {
        const int ky = t / p.kw, kx = t - (t / p.kw) * p.kw;
        const int tap_off = ky * PW + kx;
#pragma unroll
        for (int q = 0; q < CC / 2; ++q) {
#pragma unroll
            for (int b = 0; b < MB; ++b) oa[q][b] = atile[a_base[b] + tap_off + 2 * q * plane + z];
#pragma unroll
            for (int i = 0; i < NBLK; ++i) ob[q][i] = cur[(2 * q + half) * BN + 32 * i + l32 + z];
        }
    };
    // Keep a stage's matrix products where they are issued: they touch no
    // memory, so without this the compiler gathers several stages' operands
    // (and their registers) before issuing any.  The empty volatile asm stays
    // in order with the barriers', and takes the accumulators as operands.
    auto mma = [&](OpsA &oa, OpsB &ob) __attribute__((always_inline)) {
#pragma unroll
        for (int q = 0; q < CC / 2; ++q)
#pragma unroll
            for (int i = 0; i < NBLK; ++i)
#pragma unroll
                for (int b = 0; b < MB; ++b) acc[b][i] = mfma_fp4(oa[q][b], ob[q][i], acc[b][i]);
#pragma unroll
        for (int b = 0; b < MB; ++b)
#pragma unroll
            for (int i = 0; i < NBLK; ++i) asm volatile("" : "+a"(acc[b][i]));
    };

    // One stage: this wave's DMA of stage s has landed once at most the two
    // later stages' instructions are outstanding; after the barrier every
    // wave's has, and the slot of stage s-1 is free for stage s+3.  At a
    // chunk's first tap the chunk is widened first (the barrier before it
    // also retires every wave's reads of the previous chunk).
    auto stage = [&](int s, const u32x4 *cur, u32x4 *refill, OpsA &oa, OpsB &ob, OpsA &pa,
                     OpsB &pb, bool first) __attribute__((always_inline)) {
        const int ch = s / taps, t = s - ch * taps;
        wait_vmcnt<2 * kDmaPerWave>();
        if (t == 0) {
            const int z = lds_barrier();     // the A tile is free (and the region landed)
            widen_chunk(ch * CC, z);
        }
        const int z = lds_barrier();
        issue_b(s + 3, refill);
        load_ops(t, cur, z, oa, ob);
        if (!first) mma(pa, pb);
    };
    // Stage 0 alone, then four stages per iteration (the slot of a stage is
    // fixed by s % 4, its register buffer by s % 2), then the one to three
    // left over under uniform branches, then the last stage's products.
    stage(0, bslot0, bslot3, oa0, ob0, oa1, ob1, true);
    int s = 1;
    for (; s + 4 <= stages; s += 4) {
        stage(s, bslot1, bslot0, oa1, ob1, oa0, ob0, false);
        stage(s + 1, bslot2, bslot1, oa0, ob0, oa1, ob1, false);
        stage(s + 2, bslot3, bslot2, oa1, ob1, oa0, ob0, false);
        stage(s + 3, bslot0, bslot3, oa0, ob0, oa1, ob1, false);
    }
    if (s < stages) stage(s, bslot1, bslot0, oa1, ob1, oa0, ob0, false);
    if (s + 1 < stages) stage(s + 1, bslot2, bslot1, oa0, ob0, oa1, ob1, false);
    if (s + 2 < stages) stage(s + 2, bslot3, bslot2, oa1, ob1, oa0, ob0, false);
    {
        // the last stage's operands sit in buffer (stages - 1) % 2
        const bool odd = (stages - 1) & 1;
        OpsA fa;
        OpsB fb;
#pragma unroll
        for (int q = 0; q < CC / 2; ++q) {
#pragma unroll
            for (int b = 0; b < MB; ++b) fa[q][b] = odd ? oa1[q][b] : oa0[q][b];
#pragma unroll
            for (int i = 0; i < NBLK; ++i) fb[q][i] = odd ? ob1[q][i] : ob0[q][i];
        }
        mma(fa, fb);
    }
    wait_vmcnt<0>();   // the trailing prefetches land before the workgroup ends
    const int nblk = min(NBLK, (p.coutp - n_base) >> 5);

    // ---- epilogue: accumulator value v of block (b, i) is pixel
    // (v/4)*8 + half*4 + v%4 of pixel block b and filter n_base + 32i + l32.
#pragma unroll
    for (int i = 0; i < NBLK; ++i) {
        if (i >= nblk) break;
        const int co = n_base + 32 * i + l32;
        const bool co_ok = co < p.cout;
#pragma unroll
        for (int b = 0; b < MB; ++b) {
            const int mw = m0 + (wave * MB + b) * 32;
            if constexpr (OUT == OUT_BITS) {
                const float T = co_ok ? thr_to_dot_bound_f(ep_a[i], p.lo, p.hi) : -INFINITY;
                // (no flip mask: a separate instance without the XOR chain)
                const uint32_t word =
                    p.flip ? block_bits(acc[b][i], T, block_flip(p.flip, (n_base >> 5) + i, co_ok))
                           : block_bits(acc[b][i], T, 0);
                const int m = mw + lane;
                if (lane < 32 && m < p.m)
                    reinterpret_cast<uint32_t *>(p.out)[(size_t)m * p.cwo + (co >> 5)] = word;
            } else {
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int m = mw + (v >> 2) * 8 + half * 4 + (v & 3);
                    const int c = min(max((int)acc[b][i][v], p.lo), p.hi);
                    if (co_ok && m < p.m) {
                        if constexpr (OUT == OUT_FLOAT)
                            reinterpret_cast<float *>(p.out)[(size_t)m * p.cout + co] =
                                __builtin_fmaf((float)c, ep_a[i], ep_b[i]);
                        else
                            reinterpret_cast<int32_t *>(p.out)[(size_t)m * p.cout + co] = c;
                    }
                }
            }
        }
    }
}

// K-split schedule, for layers whose output tile per workgroup is small
// next to K (few pixels, many channels).  The four waves of a workgroup
// compute the same 32*MBW pixels x 32*NBLK filters, each over a quarter of
// the K steps (one K step = one tap and one pair of packed words = 64
// channels), and add their partial sums at the end.
//   * A: every packed word of the input region is widened into LDS once,
//     up front (cwe planes of the region), so any wave can take any K step.
//   * B: each wave loads the widened filters of its own K steps straight
//     into registers, kRing - 1 steps ahead; the waves never wait for each
//     other inside the loop.
//   * Reduction: every wave hands its partial sums of the blocks another
//     wave owns to that wave through LDS in one exchange (block j belongs to
//     wave j % 4); the owner adds them (fp32 adds of integers below 2^24 are
//     exact in any order) and applies the output transform.
constexpr int kRing = 4;

template <int OUT, int NBLK, int MBW>
__global__ __launch_bounds__(kMfmaThreads) void bconv2d_mfma_ks_kernel(MfmaParams p) {
    constexpr int BN = 32 * NBLK;
    constexpr int BM = 32 * MBW;
    constexpr int kBlocks = MBW * NBLK;
    extern __shared__ __attribute__((aligned(16))) u32x4 smem[];
    const int tid = threadIdx.x;
    const int lane = tid & 63, half = lane >> 5, l32 = lane & 31;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int m0 = blockIdx.x * BM;
    const int n_base = blockIdx.y * BN;
    const int cwh = p.cwe >> 1;
    const int ksteps = p.kh * p.kw * cwh;
    const int TR = p.tile_rows, PW = p.pw, plane = TR * PW;
    u32x4 *atile = smem;                                 // [cwe][TR][PW] e2m1

    int row0, col0;
    mfma_pixel(p, m0, row0, col0);
    int a_lane[MBW];                                     // this lane's A offset per pixel block
#pragma unroll
    for (int b = 0; b < MBW; ++b) {
        const int mp = min(m0 + b * 32 + l32, p.m - 1);
        int prow, pcol;
        mfma_pixel(p, mp, prow, pcol);
        a_lane[b] = half * plane + (prow - row0) * PW + pcol;
    }

    // output-transform parameters of the NBLK filter blocks
    float ep_a[NBLK], ep_b[NBLK];
#pragma unroll
    for (int i = 0; i < NBLK; ++i) {
        const int co = min(n_base + 32 * i + l32, p.cout - 1);
        if constexpr (OUT == OUT_BITS) {
            ep_a[i] = p.thr[co];
            ep_b[i] = 0.0f;
        } else if constexpr (OUT == OUT_FLOAT) {
            ep_a[i] = p.mult ? p.mult[co] : 1.0f;
            ep_b[i] = p.bias ? p.bias[co] : 0.0f;
        } else {
            ep_a[i] = ep_b[i] = 0.0f;
        }
    }

    // B of this wave's local step i (K step wave + 4i, clamped: steps past
    // the last re-read it): word row t*cwe + 2*jp + half, NBLK blocks of 32
    // filters, 16 bytes per lane per block.
    const u32x4 *wcol[NBLK];
#pragma unroll
    for (int ib = 0; ib < NBLK; ++ib)
        wcol[ib] = p.wexp + (size_t)half * p.coutp + min(n_base + 32 * ib + l32, p.coutp - 1);
    auto load_b = [&](int i, u32x4 (&dst)[NBLK]) __attribute__((always_inline)) {
        const int ks = min(wave + 4 * i, ksteps - 1);
        const int t = (int)fast_div((uint32_t)ks, p.div_cwh);
        const int jp = ks - t * cwh;
        const size_t row = (size_t)(t * p.cwe + 2 * jp) * p.coutp;
#pragma unroll
        for (int ib = 0; ib < NBLK; ++ib) dst[ib] = wcol[ib][row];
    };
    u32x4 ring[kRing][NBLK];
#pragma unroll
    for (int r = 0; r < kRing - 1; ++r) load_b(r, ring[r]);

    // ---- widen the whole region: element e = rc * groups + g holds words
    // [g*V, g*V + V) of location rc; padding locations are 0 words (+1.0),
    // or 0.0 under zero padding; words past Cw are +1.0 (their filter
    // values are 0.0).  Loads are unconditional (padding reads zeros), four
    // per thread in flight.
    {
        constexpr int U = 4;
        const int V = p.region_vec;
        const int groups = p.div_groups.d;
        const int total = plane * groups;
        for (int e0 = 0; e0 < total; e0 += U * kMfmaThreads) {
            u32x4 v[U];
            int dst[U];
            uint32_t luts[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int e = min(e0 + u * kMfmaThreads + tid, total - 1);
                const int rc = (int)fast_div((uint32_t)e, p.div_groups);
                const int g = e - rc * groups;
                const int r = (int)fast_div((uint32_t)rc, p.div_pw);
                const int c = rc - r * PW;
                const int R = row0 + r;
                const int img = (int)fast_div((uint32_t)R, p.div_ph);
                const int yy = R - img * p.ph - p.pt, xx = c - p.pl;
                const bool inside = img < p.n && (unsigned)yy < (unsigned)p.h &&
                                    (unsigned)xx < (unsigned)p.w;
                const bool load = inside && g * V < p.cw;
                const uint32_t *src =
                    load ? p.x + (((size_t)img * p.h + yy) * p.w + xx) * p.cw + g * V
                         : g_mfma_zero;
                if (V == 4)
                    v[u] = *reinterpret_cast<const u32x4 *>(src);
                else
                    v[u] = u32x4{*src, 0u, 0u, 0u};
                dst[u] = g * V * plane + rc;
                luts[u] = (p.pad_zero && !inside) ? 0u : kFp4PlusMinusLut;
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (e0 + u * kMfmaThreads + tid >= total) continue;
                if (V == 4) {
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        atile[dst[u] + j * plane] = widen_word(v[u][j], luts[u]);
                } else {
                    atile[dst[u]] = widen_word(v[u][0], luts[u]);
                }
            }
        }
    }
    int z = lds_barrier();                               // the A planes are complete

    mfma_v16f acc[MBW][NBLK];
#pragma unroll
    for (int b = 0; b < MBW; ++b)
#pragma unroll
        for (int i = 0; i < NBLK; ++i)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[b][i][v] = 0.0f;

    // A operands of local step i (clamped like the filters), double-buffered
    // in registers: step i reads the A of step i+1 before issuing its own
    // matrix products, so that the LDS latency hides behind them.
    auto load_a = [&](int i, u32x4 (&dst)[MBW]) __attribute__((always_inline)) {
        const int ks = min(wave + 4 * i, ksteps - 1);
        const int t = (int)fast_div((uint32_t)ks, p.div_cwh);
        const int jp = ks - t * cwh;
        const int ky = (int)fast_div((uint32_t)t, p.div_kw);
        const int off = 2 * jp * plane + ky * PW + (t - ky * p.kw) + z;
#pragma unroll
        for (int b = 0; b < MBW; ++b) dst[b] = atile[a_lane[b] + off];
    };
    u32x4 abuf[2][MBW];
    load_a(0, abuf[0]);

    // Local step i with its filters in `cur` and its A in `acur`; the ring
    // entry of step i-1 (`next`) takes step i + kRing - 1.
    auto step = [&](int i, u32x4 (&cur)[NBLK], u32x4 (&next)[NBLK], u32x4 (&acur)[MBW],
                    u32x4 (&anext)[MBW]) __attribute__((always_inline)) {
        load_b(i + kRing - 1, next);
        load_a(i + 1, anext);
#pragma unroll
        for (int ib = 0; ib < NBLK; ++ib)
#pragma unroll
            for (int b = 0; b < MBW; ++b) acc[b][ib] = mfma_fp4(acur[b], cur[ib], acc[b][ib]);
#pragma unroll
        for (int b = 0; b < MBW; ++b)
#pragma unroll
            for (int ib = 0; ib < NBLK; ++ib) asm volatile("" : "+a"(acc[b][ib]));
    };
    const int nsteps = ksteps > wave ? (ksteps - wave + 3) >> 2 : 0;
    int i = 0;
    for (; i + kRing <= nsteps; i += kRing) {
#pragma unroll
        for (int u = 0; u < kRing; ++u)
            step(i + u, ring[u], ring[(u + kRing - 1) % kRing], abuf[u % 2], abuf[(u + 1) % 2]);
    }
#pragma unroll
    for (int u = 0; u < kRing - 1; ++u)
        if (i + u < nsteps)
            step(i + u, ring[u], ring[(u + kRing - 1) % kRing], abuf[u % 2], abuf[(u + 1) % 2]);

    // ---- reduction: block j belongs to wave j % 4.  Every other wave stores
    // its partial sums of block j into a slot of its own (slot = (writer -
    // owner - 1) % 4, 0..2), four values per lane as one 16-byte row:
    // red[((j*3 + slot)*4 + v/4)*64 + lane] = values 4(v/4) .. +3; after one
    // barrier each owner adds its blocks' three partials.
    typedef float f32x4 __attribute__((ext_vector_type(4)));
    f32x4 *red = reinterpret_cast<f32x4 *>(smem);
    z = lds_barrier();                                   // every wave is done with the A planes
#pragma unroll
    for (int j = 0; j < kBlocks; ++j) {
        const int owner = j & 3;
        if (owner == wave) continue;
        const int slot = (wave - owner - 1) & 3;
#pragma unroll
        for (int vq = 0; vq < 4; ++vq) {
            const mfma_v16f &a = acc[j / NBLK][j % NBLK];
            red[((j * 3 + slot) * 4 + vq) * 64 + lane + z] =
                f32x4{a[4 * vq], a[4 * vq + 1], a[4 * vq + 2], a[4 * vq + 3]};
        }
    }
    z = lds_barrier();
#pragma unroll
    for (int j = 0; j < kBlocks; ++j) {
        if ((j & 3) != wave) continue;
#pragma unroll
        for (int slot = 0; slot < 3; ++slot)
#pragma unroll
            for (int vq = 0; vq < 4; ++vq) {
                const f32x4 r = red[((j * 3 + slot) * 4 + vq) * 64 + lane + z];
#pragma unroll
                for (int e = 0; e < 4; ++e) acc[j / NBLK][j % NBLK][4 * vq + e] += r[e];
            }
    }

    // ---- epilogue on this wave's blocks.  Value v of block (b, ib) is
    // pixel (v/4)*8 + half*4 + v%4 of pixel block b and filter
    // n_base + 32*ib + l32.
    const int nblk = min(NBLK, (p.coutp - n_base) >> 5);
#pragma unroll
    for (int j = 0; j < kBlocks; ++j) {
        if ((j & 3) != wave) continue;
        const int b = j / NBLK, ib = j % NBLK;
        if (ib >= nblk) continue;
        const mfma_v16f val = acc[b][ib];
        const int co = n_base + 32 * ib + l32;
        const bool co_ok = co < p.cout;
        const int mw = m0 + b * 32;
        if constexpr (OUT == OUT_BITS) {
            const float T = co_ok ? thr_to_dot_bound_f(ep_a[ib], p.lo, p.hi) : -INFINITY;
            const uint32_t word =
                p.flip ? block_bits(val, T, block_flip(p.flip, (n_base >> 5) + ib, co_ok))
                       : block_bits(val, T, 0);
            const int m = mw + lane;
            if (lane < 32 && m < p.m)
                reinterpret_cast<uint32_t *>(p.out)[(size_t)m * p.cwo + (co >> 5)] = word;
        } else {
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int m = mw + (v >> 2) * 8 + half * 4 + (v & 3);
                const int c = min(max((int)val[v], p.lo), p.hi);
                if (co_ok && m < p.m) {
                    if constexpr (OUT == OUT_FLOAT)
                        reinterpret_cast<float *>(p.out)[(size_t)m * p.cout + co] =
                            __builtin_fmaf((float)c, ep_a[ib], ep_b[ib]);
                    else
                        reinterpret_cast<int32_t *>(p.out)[(size_t)m * p.cout + co] = c;
                }
            }
        }
    }
}

// Filters widened once per filter tensor into the B layout:
//   wexp[(t*CwE + j)*CoutP + co] = 32 e2m1 codes of word j of tap t of
//   filter co; channels past C_in, words past Cw and filters past Cout are
//   0.0 (they then add nothing to any dot).
__global__ __launch_bounds__(256) void mfma_expand_weights_kernel(const uint32_t *__restrict__ w,
                                                                  u32x4 *__restrict__ wexp,
                                                                  int cout, int coutp, int taps,
                                                                  int cw, int cwe, int cin) {
    const int64_t total = (int64_t)taps * cwe * coutp;
    for (int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * 256) {
        const int64_t k = idx / coutp;
        const int co = (int)(idx - k * coutp);
        const int t = (int)(k / cwe), j = (int)(k - (int64_t)t * cwe);
        u32x4 o = {0u, 0u, 0u, 0u};
        if (co < cout && j < cw) {
            const uint32_t bits = w[((size_t)co * taps + t) * cw + j];
            const int nvalid = min(32, cin - 32 * j);
            const uint32_t valid = nvalid >= 32 ? 0xFFFFFFFFu : (1u << nvalid) - 1u;
            o = widen_word(bits, kFp4PlusMinusLut) & widen_word(valid, kFp4ValidLut);
        }
        wexp[idx] = o;
    }
}

}  // namespace lce
