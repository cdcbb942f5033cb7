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

// e2m1 codes: +1.0 = 0x2, -1.0 = 0xA (the sign is bit 3 of the nibble).
// A widened word fills all eight nibbles of each 32-bit lane word with
// +1.0 before the sign bits are ORed in; zero padding fills them with 0.0.
constexpr uint32_t kFp4PlusOne = 0x22222222u;
constexpr uint32_t kFp4SignBits = 0x88888888u;

// K steps (S*KS) a filter-stationary instance covers at most.
constexpr int kFsMaxSteps = 72;

struct MfmaParams {
    const uint32_t *x;      // [N][H][W][Cw] bitpacked activations
    const u32x4 *wexp;      // [KH*KW*CwE][CoutP] widened filters (16 bytes = 32 values)
    const uint32_t *wpk;    // [KH*KW*CwE][CoutP] the same filters packed (4 bytes = 32 values)
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
    int32_t fs_pixels;               // output pixels per workgroup (filter-stationary)
    int32_t fs_thr_off;              // filter-stationary: float offset of the bounds in LDS
                                     // from the end of the A tile
    int32_t pad_zero;                // 1: padded locations are 0.0
    int32_t region_vec;              // words per lane per load when staging the region: 4 or 1
    FastDiv div_ohw, div_ow, div_ph, div_pw;
    FastDiv div_plane;               // tile_rows * pw: region locations
    FastDiv div_cwh, div_kw;         // cwe / 2 (word pairs per tap), kw
    FastDiv div_groups;              // region_vec-word groups per location
    FastDiv div_ks_gx;               // K-split schedule: pixel tiles (grid x)
    // filter-stationary schedules: A-tile offset (in 16-byte words) of K step
    // s = (tap t = ky*KW + kx, word pair q) from a pixel's window origin,
    // 2q*plane + ky*PW + kx (plane = tile_rows*pw), in bits 0-23, and the
    // number of real channels in the step's word pair, min(64, C_in - 64q),
    // in bits 24-31; steps past the last repeat the last one
    int32_t fs_koff[kFsMaxSteps];
};

typedef int mfma_v8i __attribute__((ext_vector_type(8)));
typedef float mfma_v16f __attribute__((ext_vector_type(16)));


// Packed word -> 32 e2m1 codes (16 bytes).  The order of k inside an MFMA
// operand is free as long as both operands use the same one, so channel c of
// the word goes where it is cheapest: 32-bit word c % 4, nibble c / 4.  Then
// word d of the result is the packed word shifted so that channels d, d+4,
// ... land on the nibbles' sign bits, masked, over a field of +1.0 codes:
// two ALU operations per 32-bit word.  `fill` is kFp4PlusOne (bit 0 -> +1.0,
// bit 1 -> -1.0), or 0 for an all-0.0 location (zero padding; its bits are 0).
__device__ __forceinline__ u32x4 widen_word(uint32_t w, uint32_t fill) {
    u32x4 o;
    o.x = ((w << 3) & kFp4SignBits) | fill;
    o.y = ((w << 2) & kFp4SignBits) | fill;
    o.z = ((w << 1) & kFp4SignBits) | fill;
    o.w = (w & kFp4SignBits) | fill;
    return o;
}

// widen_word with the sign-bit mask in a register (mask = kFp4SignBits held
// in a VGPR): each 32-bit word is then one shift and one AND-OR, since a
// VALU instruction here takes at most one scalar or literal operand and the
// fill is scalar.
__device__ __forceinline__ u32x4 widen_word_vm(uint32_t w, uint32_t fill, uint32_t mask) {
    u32x4 o;
    o.x = ((w << 3) & mask) | fill;
    o.y = ((w << 2) & mask) | fill;
    o.z = ((w << 1) & mask) | fill;
    o.w = (w & mask) | fill;
    return o;
}

// Mask of the nibbles a widened word may keep: nibble c/4 of 32-bit word
// c % 4 is 0xF for every channel c whose bit is set in `valid`.
__device__ __forceinline__ u32x4 widen_valid_mask(uint32_t valid) {
    u32x4 o;
    o.x = (((valid << 3) & kFp4SignBits) >> 3) * 0xFu;
    o.y = (((valid << 2) & kFp4SignBits) >> 3) * 0xFu;
    o.z = (((valid << 1) & kFp4SignBits) >> 3) * 0xFu;
    o.w = ((valid & kFp4SignBits) >> 3) * 0xFu;
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

// Output bits of value V of an accumulator block (see block_bits): the
// lane mask `m` of "value < T" holds pixels r0 (lanes 0-31) and r0 + 4
// (lanes 32-63), r0 = (V/4)*8 + V%4, and two v_writelane drop them into the
// lanes of their pixels.  A v_writelane that reads the mask of a compare
// issued right before it stalls the wave until the compare's SGPR write
// lands (measured: ~35 cycles per value next to LDS reads), so callers
// issue the compares well ahead.  The s_nop 1 covers a VALU-written SGPR in
// any case (the compiler's hazard recognizer does not look inside inline
// asm).
template <int V>
__device__ __forceinline__ void write_value_bits(uint64_t m, uint32_t &word) {
    constexpr int r0 = (V >> 2) * 8 + (V & 3);
    asm volatile(
        "s_nop 1\n\t"
        "v_writelane_b32 %0, %1, %3\n\t"
        "v_writelane_b32 %0, %2, %4"
        : "+v"(word)
        : "s"((uint32_t)m), "s"((uint32_t)(m >> 32)), "i"(r0), "i"(r0 + 4));
}

// Bitpacked output of one 32x32 accumulator block (pixel-split schedule).
// Value v of the block is pixel (v/4)*8 + half*4 + v%4 and filter
// lane % 32, so one ballot of
// "value < T" over the wave gives the 32 filter bits of two pixels (lanes
// 0-31 and 32-63); v_writelane drops each 32-bit half into the lane of its
// pixel.  fmask (wave-uniform) flips chosen filters.  Lane l < 32 returns
// the word of pixel l.  All sixteen compares come first, so that no
// v_writelane waits for the compare right before it, and the lane writes
// alternate between four partial words (consecutive writes to one register
// form a dependent chain).
template <int... V>
__device__ __forceinline__ uint32_t block_bits_impl(const mfma_v16f &val, float T,
                                                    uint64_t fmask,
                                                    std::integer_sequence<int, V...>) {
    uint64_t m[16];
    ((m[V] = __ballot(val[V] < T) ^ fmask), ...);
    uint32_t w[4] = {0u, 0u, 0u, 0u};
    (write_value_bits<V>(m[V], w[V & 3]), ...);
    return (w[0] | w[1]) | (w[2] | w[3]);
}
__device__ __forceinline__ uint32_t block_bits(const mfma_v16f &val, float T, uint64_t fmask) {
    return block_bits_impl(val, T, fmask, std::make_integer_sequence<int, 16>{});
}

// Every cache line of the kernel arguments up to the K-split grid divisor
// (one field per 64-byte line), fetched in one round trip at the top of a
// kernel: the compiler would otherwise load the fields in several dependent
// batches (behind branches), each first touch of a line a full memory
// latency.
__device__ __forceinline__ void fetch_arg_lines(const MfmaParams &p) {
    asm volatile("" ::"s"(p.x), "s"(p.oh), "s"(p.m), "s"(p.div_pw.d), "s"(p.div_ks_gx.d));
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
    fetch_arg_lines(p);
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
            uint32_t fill = kFp4PlusOne;
            if (p.pad_zero) {
                const int r = (int)fast_div((uint32_t)rc, p.div_pw);
                const int xx = rc - r * PW - p.pl;
                if (!(rowok[r + z] && (unsigned)xx < (unsigned)p.w)) fill = 0u;
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
            for (int j = 0; j < CC; ++j) atile[j * plane + rc] = widen_word(bits[j], fill);
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

// Whether region location rc lies inside the image.  The region is
// tile_rows x pw locations from padded row row0 and padded column c0 (c0 = 0
// unless a filter-stationary workgroup stages only its share's window of
// columns, pw then being the window's width).
__device__ __forceinline__ bool region_inside(const MfmaParams &p, int row0, int c0, int rc) {
    const int r = (int)fast_div((uint32_t)rc, p.div_pw);
    const int c = c0 + rc - r * p.pw;
    const int R = row0 + r;
    const int img = (int)fast_div((uint32_t)R, p.div_ph);
    const int yy = R - img * p.ph - p.pt, xx = c - p.pl;
    return img < p.n && (unsigned)yy < (unsigned)p.h && (unsigned)xx < (unsigned)p.w;
}

// A copy of the parameters whose geometry fields (the ones the region
// staging and the pixel arithmetic read) are held in scalar registers: each
// passes through an empty asm statement, so the compiler keeps the value
// instead of reloading it from the kernel arguments wherever it is used (it
// treats argument loads as free to repeat, and each repeat is a dependent
// scalar-cache round trip in the set-up).
__device__ __forceinline__ MfmaParams pinned_geometry(const MfmaParams &p) {
    MfmaParams q = p;
    asm volatile("" : "+s"(q.n), "+s"(q.h), "+s"(q.w), "+s"(q.cw), "+s"(q.cwe), "+s"(q.pw),
                      "+s"(q.ph), "+s"(q.pt), "+s"(q.pl), "+s"(q.sh), "+s"(q.sw), "+s"(q.ow),
                      "+s"(q.region_vec), "+s"(q.pad_zero), "+s"(q.m));
    asm volatile("" : "+s"(q.div_plane.d), "+s"(q.div_plane.magic), "+s"(q.div_plane.shift),
                      "+s"(q.div_pw.d), "+s"(q.div_pw.magic), "+s"(q.div_pw.shift),
                      "+s"(q.div_ph.d), "+s"(q.div_ph.magic), "+s"(q.div_ph.shift),
                      "+s"(q.div_ohw.d), "+s"(q.div_ohw.magic), "+s"(q.div_ohw.shift),
                      "+s"(q.div_ow.magic), "+s"(q.div_ow.shift));
    return q;
}

// Buffer resources (gfx9 raw buffers: base, byte size, no stride; the
// fourth descriptor word selects 32-bit data).  A buffer load takes a
// wave-uniform base and byte offset in scalar registers and a 32-bit lane
// offset; offsets at or past the size read zeros, which the region loads
// use for padding locations.  The host keeps every buffer below 2^31 bytes.
constexpr int kBufDword3 = 0x00020000;
constexpr int kBufOutside = (int)0x80000000u;      // a lane offset past any buffer

__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_of(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes,
                                             kBufDword3);
}

// the bitpacked input as a buffer
__device__ __forceinline__ __amdgpu_buffer_rsrc_t input_buffer(const MfmaParams &p) {
    return buffer_of(p.x, (uint32_t)p.n * p.h * p.w * p.cw * 4u);
}

// the widened (16 bytes per element) or packed (4 bytes) filters as a buffer
__device__ __forceinline__ __amdgpu_buffer_rsrc_t filter_buffer(const MfmaParams &p, bool packed) {
    const uint32_t elems = (uint32_t)p.kh * p.kw * p.cwe * p.coutp;
    return packed ? buffer_of(p.wpk, elems * 4u) : buffer_of(p.wexp, elems * 16u);
}

// The packed region staged through registers (filter-stationary and K-split
// schedules): each thread loads up to kRegU elements (an element is
// region_vec words of one location), widens them in registers and writes
// them to the A tile once (atile[j*plane + rc] = word j of location rc),
// with no LDS round trip and no barrier in between.  region_load issues one
// chunk's buffer loads (the caller issues its filter loads after it, so
// that both latencies overlap; the compiler waits for the region words where
// region_widen first uses them); a padding location's lane offset lies past
// the input, so it reads zeros, and it is flagged in `out`.
constexpr int kRegU = 4;

struct RegionChunk {
    u32x4 w[kRegU];
    uint32_t out;                        // bit u: element u lies outside the image
};

// byte offset in the input of word `word` of region location rc
// (kBufOutside when the location is outside the image; region origin as in
// region_inside)
__device__ __forceinline__ int region_offset(const MfmaParams &p, int row0, int c0, int rc,
                                             int word, bool &inside) {
    const int r = (int)fast_div((uint32_t)rc, p.div_pw);
    const int c = c0 + rc - r * p.pw;
    const int R = row0 + r;
    const int img = (int)fast_div((uint32_t)R, p.div_ph);
    const int yy = R - img * p.ph - p.pt, xx = c - p.pl;
    inside = img < p.n && (unsigned)yy < (unsigned)p.h && (unsigned)xx < (unsigned)p.w;
    const uint32_t w = (((uint32_t)img * (uint32_t)p.h + (uint32_t)yy) * (uint32_t)p.w +
                        (uint32_t)xx) * (uint32_t)p.cw + (uint32_t)word;
    return inside ? (int)(w * 4u) : kBufOutside;
}

// elements of the region: plane * Cw / region_vec
__device__ __forceinline__ int region_elements(const MfmaParams &p, int plane) {
    return p.region_vec == 4 ? plane * (p.cw >> 2) : plane * p.cw;
}

template <int NT>
__device__ __forceinline__ void region_load(const MfmaParams &p, int row0, int c0, int plane,
                                            int tid, int e0, RegionChunk &ch) {
    const int total = region_elements(p, plane);
    const __amdgpu_buffer_rsrc_t xb = input_buffer(p);
    ch.out = 0;
    // (slots whose whole wave lies past the region are skipped, a uniform
    // branch, and hold zeros)
    const int wave_e0 = e0 + (tid & ~63);
    if (p.region_vec == 4) {
#pragma unroll
        for (int u = 0; u < kRegU; ++u) {
            if (wave_e0 + u * NT >= total) {
                ch.w[u] = u32x4{0u, 0u, 0u, 0u};
                continue;
            }
            const int e = min(e0 + u * NT + tid, total - 1);
            const int g = (int)fast_div((uint32_t)e, p.div_plane);
            bool in;
            const int off = region_offset(p, row0, c0, e - g * plane, 4 * g, in);
            ch.w[u] = __builtin_amdgcn_raw_buffer_load_b128(xb, off, 0, 0);
            ch.out |= in ? 0u : 1u << u;
        }
    } else {
#pragma unroll
        for (int u = 0; u < kRegU; ++u) {
            if (wave_e0 + u * NT >= total) {
                ch.w[u] = u32x4{0u, 0u, 0u, 0u};
                continue;
            }
            const int e = min(e0 + u * NT + tid, total - 1);
            const int j = (int)fast_div((uint32_t)e, p.div_plane);
            bool in;
            const int off = region_offset(p, row0, c0, e - j * plane, j, in);
            ch.w[u].x = __builtin_amdgcn_raw_buffer_load_b32(xb, off, 0, 0);
            ch.out |= in ? 0u : 1u << u;
        }
    }
}

// Widen a loaded chunk into the A tile: +1.0/-1.0 from the bits, 0.0 at
// padding locations under zero padding.
template <int NT>
__device__ __forceinline__ void region_widen(const MfmaParams &p, const RegionChunk &ch,
                                             u32x4 *atile, int plane, int tid, int e0) {
    const int total = region_elements(p, plane);
#pragma unroll
    for (int u = 0; u < kRegU; ++u) {
        const int e = e0 + u * NT + tid;
        if (e >= total) break;
        const uint32_t fill = p.pad_zero && ((ch.out >> u) & 1u) ? 0u : kFp4PlusOne;
        if (p.region_vec == 4) {
            const int g = (int)fast_div((uint32_t)e, p.div_plane);
            const int rc = e - g * plane;
#pragma unroll
            for (int k = 0; k < 4; ++k) atile[(4 * g + k) * plane + rc] = widen_word(ch.w[u][k], fill);
        } else {
            atile[e] = widen_word(ch.w[u].x, fill);
        }
    }
}

// The rest of the A tile after the first chunk (regions of more than
// kRegU*NT elements: load, wait, widen), then the words past Cw: +1.0, or
// 0.0 outside the image under zero padding.
template <int NT>
__device__ __forceinline__ void region_finish(const MfmaParams &p, u32x4 *atile, int row0,
                                              int c0, int plane, int tid) {
    const int total = region_elements(p, plane);
    for (int e0 = kRegU * NT; e0 < total; e0 += kRegU * NT) {
        RegionChunk ch;
        region_load<NT>(p, row0, c0, plane, tid, e0, ch);
        region_widen<NT>(p, ch, atile, plane, tid, e0);
    }
    for (int e = plane * p.cw + tid; e < plane * p.cwe; e += NT) {
        uint32_t fill = kFp4PlusOne;
        if (p.pad_zero) {
            const int j = (int)fast_div((uint32_t)e, p.div_plane);
            if (!region_inside(p, row0, c0, e - j * plane)) fill = 0u;
        }
        atile[e] = widen_word(0u, fill);
    }
}

// LceQuantize fused into the region staging (arXiv 2011.09398 Section 3.2:
// a float activation is sign-binarized, then convolved).  The input is
// float32 NHWC with C_in a multiple of 32, and p.x points at it.  An element
// is word j of region location rc, i.e. channels 32j .. 32j+31 of that
// location: 128 bytes, eight 16-byte buffer loads.  Its bit c is x < 0 (the
// sign test of the bitpack kernel: -0.0 and NaN give +1), and it is then
// widened like a packed word.  A location outside the image reads zeros past
// the buffer, which binarize to +1.0 (one padding); zero padding takes the
// outside flag, as for packed input.  The host keeps the float input below
// 2 GiB.
typedef float f32x4_t __attribute__((ext_vector_type(4)));
constexpr int kRegUF = 2;

struct RegionChunkF {
    f32x4_t v[kRegUF][8];
    uint32_t out;                        // bit u: element u lies outside the image
};

template <int NT>
__device__ __forceinline__ void region_load_f(const MfmaParams &p, int row0, int c0, int plane,
                                              int tid, int e0, RegionChunkF &ch) {
    const int total = plane * p.cw;
    const __amdgpu_buffer_rsrc_t xb =
        buffer_of(p.x, (uint32_t)p.n * p.h * p.w * p.cw * 128u);
    ch.out = 0;
    const int wave_e0 = e0 + (tid & ~63);
#pragma unroll
    for (int u = 0; u < kRegUF; ++u) {
        if (wave_e0 + u * NT >= total) {
#pragma unroll
            for (int i = 0; i < 8; ++i) ch.v[u][i] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
            continue;
        }
        const int e = min(e0 + u * NT + tid, total - 1);
        const int j = (int)fast_div((uint32_t)e, p.div_plane);
        bool in;
        // byte offset of packed word j of the location, times 32: its floats
        const int off = region_offset(p, row0, c0, e - j * plane, j, in);
        const int offf = in ? off * 32 : kBufOutside;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const auto w = __builtin_amdgcn_raw_buffer_load_b128(xb, offf + 16 * i, 0, 0);
            ch.v[u][i] = f32x4_t{__uint_as_float(w[0]), __uint_as_float(w[1]),
                                 __uint_as_float(w[2]), __uint_as_float(w[3])};
        }
        ch.out |= in ? 0u : 1u << u;
    }
}

template <int NT>
__device__ __forceinline__ void region_widen_f(const MfmaParams &p, const RegionChunkF &ch,
                                               u32x4 *atile, int plane, int tid, int e0) {
    const int total = plane * p.cw;
#pragma unroll
    for (int u = 0; u < kRegUF; ++u) {
        const int e = e0 + u * NT + tid;
        if (e >= total) break;
        uint32_t bits = 0;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const f32x4_t f = ch.v[u][i];
            const uint32_t nib = (uint32_t)(f.x < 0.0f) | ((uint32_t)(f.y < 0.0f) << 1) |
                                 ((uint32_t)(f.z < 0.0f) << 2) | ((uint32_t)(f.w < 0.0f) << 3);
            bits |= nib << (4 * i);
        }
        const uint32_t fill = p.pad_zero && ((ch.out >> u) & 1u) ? 0u : kFp4PlusOne;
        atile[e] = widen_word(bits, fill);
    }
}

// The rest of the float region after the first chunk, then the words past
// Cw (as region_finish).
template <int NT>
__device__ __forceinline__ void region_finish_f(const MfmaParams &p, u32x4 *atile, int row0,
                                                int c0, int plane, int tid) {
    const int total = plane * p.cw;
    for (int e0 = kRegUF * NT; e0 < total; e0 += kRegUF * NT) {
        RegionChunkF ch;
        region_load_f<NT>(p, row0, c0, plane, tid, e0, ch);
        region_widen_f<NT>(p, ch, atile, plane, tid, e0);
    }
    for (int e = plane * p.cw + tid; e < plane * p.cwe; e += NT) {
        uint32_t fill = kFp4PlusOne;
        if (p.pad_zero) {
            const int j = (int)fast_div((uint32_t)e, p.div_plane);
            if (!region_inside(p, row0, c0, e - j * plane)) fill = 0u;
        }
        atile[e] = widen_word(0u, fill);
    }
}

// Bitpacked output of one transposed 32x32 accumulator block (filters as
// the row operand: lane = pixel lane % 32, value v = filter (v/4)*8 +
// half*4 + v%4), given the dot bounds t[q] of filters 8q + half*4 + 0..3.
// Bit f of the returned word (the same in lanes l and l + 32) is filter f's
// "dot < T", the sign of dot - T (an integer dot below 2^24 minus an
// integer or infinite bound: exact in sign).  The signs are shifted into a
// word last value first (one v_alignbit_b32 each), so that bit v is value
// v's; nibble q then moves to nibble 2q + half and the lane halves merge.
__device__ __forceinline__ uint32_t transposed_block_bits(const mfma_v16f &val,
                                                          const float4 (&t)[4], int half) {
    uint32_t w = 0;
#pragma unroll
    for (int k = 0; k < 16; ++k) {
        const int v = 15 - k;
        const float4 tq = t[v >> 2];
        const float tv = (v & 3) == 0 ? tq.x : (v & 3) == 1 ? tq.y : (v & 3) == 2 ? tq.z : tq.w;
        const uint32_t u = __float_as_uint(val[v] - tv);
        w = k == 0 ? u >> 31 : __builtin_amdgcn_alignbit(w, u, 31);
    }
    w = (w | (w << 8)) & 0x00FF00FFu;
    w = ((w | (w << 4)) & 0x0F0F0F0Fu) << (4 * half);
    const auto sw = __builtin_amdgcn_permlane32_swap(w, w, false, false);
    return sw[0] | sw[1];
}

// K-split schedule, for layers whose output tile per workgroup is small
// next to K (few pixels, many channels).  The four waves of a workgroup
// compute the same 32*MBW pixels x 32*NBLK filters, each over a quarter of
// the K steps (one K step = one tap and one pair of packed words = 64
// channels), and add their partial sums at the end.
//   * A: every packed word of the input region is loaded into registers
//     and widened into LDS once, up front (cwe planes of the region), so
//     any wave can take any K step.
//   * B: each wave loads the widened filters of its own K steps straight
//     into registers, kRing - 1 steps ahead; the waves never wait for each
//     other inside the loop.
//   * Reduction: every wave hands its partial sums of the blocks another
//     wave owns to that wave through LDS in one exchange (block j belongs to
//     wave j % 4); the owner adds them (fp32 adds of integers below 2^24 are
//     exact in any order) and applies the output transform.
//   * Bitpacked output: the products are transposed (filters as the row
//     operand, lane = pixel), so that each lane packs its own pixel's filter
//     bits from the signs of dot - bound (transposed_block_bits), with the
//     bounds of the workgroup's filters in LDS.
//   (Loading the packed filter copy and widening it at use, as the
//   filter-stationary schedule does, measured 10% slower here.)
//   * Tiles are renumbered so that each of the 8 XCDs (which take the
//     workgroups round-robin in launch order, each with its own L2) runs a
//     contiguous range of them in filter-major order: its L2 then holds only
//     its own filter tiles.
constexpr int kRing = 4;
constexpr unsigned kXcds = 8;

// QF: the input is float32 and binarized while its region is staged
// (region_load_f), LceQuantize fused into the convolution.
template <int OUT, int NBLK, int MBW, bool QF = false>
__global__ __launch_bounds__(kMfmaThreads) void bconv2d_mfma_ks_kernel(MfmaParams p) {
    constexpr int BN = 32 * NBLK;
    constexpr int BM = 32 * MBW;
    constexpr int kBlocks = MBW * NBLK;
    extern __shared__ __attribute__((aligned(16))) u32x4 smem[];
    const int tid = threadIdx.x;
    const int lane = tid & 63, half = lane >> 5, l32 = lane & 31;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    fetch_arg_lines(p);
    int m0, n_base;
    {
        // launch index L goes to XCD L % 8 as its (L / 8)-th; XCD x runs
        // tiles [x*q + min(x, rem), ...) of the T = q*8 + rem
        const unsigned gx = gridDim.x, T = gx * gridDim.y;
        const unsigned L = blockIdx.y * gx + blockIdx.x;
        const unsigned q = T / kXcds, rem = T % kXcds, x = L % kXcds;
        const unsigned t = x * q + min(x, rem) + L / kXcds;
        const unsigned ty = fast_div(t, p.div_ks_gx);
        m0 = (int)(t - ty * gx) * BM;
        n_base = (int)ty * BN;
    }
    const int cwh = p.cwe >> 1;
    const int ksteps = p.kh * p.kw * cwh;
    const int TR = p.tile_rows, PW = p.pw, plane = TR * PW;
    u32x4 *atile = smem;                                 // [cwe][TR][PW] e2m1

    const MfmaParams g = pinned_geometry(p);     // (geometry in scalar registers)
    int row0, col0;
    mfma_pixel(g, m0, row0, col0);
    int a_lane[MBW];                                     // this lane's A offset per pixel block
#pragma unroll
    for (int b = 0; b < MBW; ++b) {
        const int mp = min(m0 + b * 32 + l32, p.m - 1);
        int prow, pcol;
        mfma_pixel(g, mp, prow, pcol);
        a_lane[b] = half * plane + (prow - row0) * PW + pcol;
    }

    // the region's first chunk (its loads before the filters': the widening
    // needs it first)
    std::conditional_t<QF, RegionChunkF, RegionChunk> rch;
    if constexpr (QF)
        region_load_f<kMfmaThreads>(g, row0, 0, plane, tid, 0, rch);
    else
        region_load<kMfmaThreads>(g, row0, 0, plane, tid, 0, rch);

    // output-transform parameters of the NBLK filter blocks (buffer loads
    // after the region's, so that its widening does not wait for them; an
    // absent array reads zeros, replaced by the default)
    float ep_a[NBLK], ep_b[NBLK];
    uint32_t flip_w[NBLK];                               // bitpacked output: flip words
    {
        const uint32_t cb = (uint32_t)p.cout * 4u;
        const __amdgpu_buffer_rsrc_t fb = buffer_of(p.flip, p.flip ? (uint32_t)p.cwo * 4u : 0u);
        const __amdgpu_buffer_rsrc_t ab = buffer_of(OUT == OUT_BITS ? p.thr : p.mult,
                                                    OUT == OUT_BITS || p.mult ? cb : 0u);
        const __amdgpu_buffer_rsrc_t bb = buffer_of(p.bias, p.bias ? cb : 0u);
#pragma unroll
        for (int i = 0; i < NBLK; ++i) {
            const int co4 = min(n_base + 32 * i + l32, p.cout - 1) * 4;
            ep_a[i] = ep_b[i] = 0.0f;
            flip_w[i] = 0u;
            if constexpr (OUT == OUT_BITS)
                flip_w[i] = __builtin_amdgcn_raw_buffer_load_b32(
                    fb, min((n_base >> 5) + i, p.cwo - 1) * 4, 0, 0);
            if constexpr (OUT == OUT_BITS) {
                ep_a[i] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(ab, co4, 0, 0));
            } else if constexpr (OUT == OUT_FLOAT) {
                const float m = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(ab, co4, 0, 0));
                const float b = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(bb, co4, 0, 0));
                ep_a[i] = p.mult ? m : 1.0f;
                ep_b[i] = p.bias ? b : 0.0f;
            }
        }
    }

    // B of this wave's local step i (K step wave + 4i, clamped: steps past
    // the last re-read it): word row t*cwe + 2*jp + half, NBLK blocks of 32
    // filters, 16 bytes per lane per block.
    // (buffer loads: lane offset of the filter column, uniform byte offset
    // of the row)
    const __amdgpu_buffer_rsrc_t wb = filter_buffer(p, false);
    int wcol[NBLK];
#pragma unroll
    for (int ib = 0; ib < NBLK; ++ib)
        wcol[ib] = (half * p.coutp + min(n_base + 32 * ib + l32, p.coutp - 1)) * 16;
    auto load_b = [&](int i, u32x4 (&dst)[NBLK]) __attribute__((always_inline)) {
        const int ks = min(wave + 4 * i, ksteps - 1);
        const int t = (int)fast_div((uint32_t)ks, p.div_cwh);
        const int jp = ks - t * cwh;
        const int row = (t * p.cwe + 2 * jp) * p.coutp * 16;
#pragma unroll
        for (int ib = 0; ib < NBLK; ++ib)
            dst[ib] = __builtin_amdgcn_raw_buffer_load_b128(wb, wcol[ib], row, 0);
    };
    u32x4 ring[kRing][NBLK];
#pragma unroll
    for (int r = 0; r < kRing - 1; ++r) load_b(r, ring[r]);

    // ---- widen the whole region (every word of every location) as its
    // words arrive, while the filter ring is still arriving
    if constexpr (QF) {
        region_widen_f<kMfmaThreads>(g, rch, atile, plane, tid, 0);
        region_finish_f<kMfmaThreads>(g, atile, row0, 0, plane, tid);
    } else {
        region_widen<kMfmaThreads>(g, rch, atile, plane, tid, 0);
        region_finish<kMfmaThreads>(g, atile, row0, 0, plane, tid);
    }
    // bitpacked output: the dot bound of each of the workgroup's filters, in
    // LDS past the A planes and the reduction buffer (tb[32*ib + f] for
    // filter n_base + 32*ib + f; filters past C_out get -inf, bit 0)
    float *tb = reinterpret_cast<float *>(
        reinterpret_cast<char *>(smem) + max(p.cwe * plane * 16, kBlocks * 3 * 16 * 64 * 4));
    if constexpr (OUT == OUT_BITS) {
        if (wave == 0 && half == 0) {
#pragma unroll
            for (int ib = 0; ib < NBLK; ++ib)
                tb[32 * ib + l32] = n_base + 32 * ib + l32 < p.cout
                                        ? thr_to_dot_bound_f(ep_a[ib], p.lo, p.hi)
                                        : -INFINITY;
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
            for (int b = 0; b < MBW; ++b) {
                if constexpr (OUT == OUT_BITS)      // transposed: lane = pixel
                    acc[b][ib] = mfma_fp4(cur[ib], acur[b], acc[b][ib]);
                else
                    acc[b][ib] = mfma_fp4(acur[b], cur[ib], acc[b][ib]);
            }
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
    // n_base + 32*ib + l32; bitpacked output (transposed products): pixel
    // l32 of block b and filter n_base + 32*ib + (v/4)*8 + half*4 + v%4.
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
            float4 t[4];
#pragma unroll
            for (int q = 0; q < 4; ++q)
                t[q] = reinterpret_cast<const float4 *>(tb + 32 * ib + 8 * q + 4 * half)[z];
            uint32_t word = transposed_block_bits(val, t, half);
            // the flip word of the block (0 without a flip mask), restricted
            // to the filters below C_out
            const int nv = p.cout - (n_base + 32 * ib);
            word ^= flip_w[ib] & (nv >= 32 ? ~0u : (1u << nv) - 1u);
            const int m = mw + l32;
            if (lane < 32 && m < p.m)
                reinterpret_cast<uint32_t *>(p.out)[(size_t)m * p.cwo + (n_base >> 5) + ib] = word;
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

// Filter-stationary schedule.  Each wave keeps the widened filters of one
// block of 32 filters for its KS K steps in registers for the whole kernel
// (16 bytes per lane per step, loaded once, from the packed copy where every
// channel is valid, and waited for step by step in the first pair); the
// workgroup loads its input region into registers (buffer loads issued
// before the filters'), widens it into LDS once, and then runs through its
// pixel blocks two at a time, reading only the A operands from LDS.
// Nothing is staged inside the loop, and the loop is software-pipelined
// across pixel-block pairs:
//   * a ring of A operands runs a few K steps ahead of the matrix products,
//     into the next pair;
//   * the previous pair is finished (partial-sum exchange and output
//     transform) in small pieces between the current pair's products, so
//     that the matrix pipe never waits for the epilogue;
//   * compiler and scheduling barriers at every K step keep that order (the
//     compiler would otherwise hoist every LDS read of a pair to its top).
// F = 4/S filter blocks per workgroup; S = 2 waves share a filter block
// when K is long, each taking KS consecutive K steps (one K step = one tap
// and one pair of packed words = 64 channels; steps past the last add 0.0
// filters).  Their partial sums meet in LDS once per pair (one barrier, two
// alternating buffers), each wave finishing one block of the pair.  The host
// gives each workgroup the same number of pixel blocks and about one
// workgroup per CU (two where a wave's filters are few).
// Ring of A operands: K step i of every pair uses slot i % D and, before
// its products, refills the slot of step i-1 with step i + D - 1 (of this
// pair, or of the next past its end), so D divides KS (6, 4 or 3 K steps,
// else KS itself) and the reads run D - 1 steps ahead.  The refill comes first
// in the step because the loop's pace is set by LDS: every read issued
// later, behind the step's other work, would leave the LDS idle meanwhile.
constexpr int fs_depth(int ks) { return ks % 6 == 0 ? 6 : ks % 4 == 0 ? 4 : ks % 3 == 0 ? 3 : ks; }

// Calls f(std::integral_constant<int, I>) for I = 0 .. N-1 in order.
template <typename Fn, int... I>
__device__ __forceinline__ void for_each_index(Fn &&f, std::integer_sequence<int, I...>) {
    (f(std::integral_constant<int, I>{}), ...);
}


// QF: the input is float32 and binarized while its region is staged
// (region_load_f), LceQuantize fused into the convolution.  WIN: every
// share lies within one output row and the workgroup stages only the padded
// columns its windows read (pw is then their count, from the share's first
// pixel's window origin); otherwise whole padded rows.
template <int KS, int S, int OUT, bool PK, bool QF = false, bool WIN = false>
__global__ __launch_bounds__(kMfmaThreads) void bconv2d_mfma_fs_kernel(MfmaParams p) {
    static_assert(S == 1 || S == 2 || S == 4, "1, 2 or 4 waves per filter block");
    // every argument line this kernel reads in one round trip, the tap
    // offsets of this wave's K steps included
    {
        const int ks0 = S == 1 ? 0 : __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6)) / (4 / S) * KS;
        fetch_arg_lines(p);
        asm volatile("" ::"s"(p.fs_koff[ks0]), "s"(p.fs_koff[ks0 + KS / 2]),
                     "s"(p.fs_koff[ks0 + KS - 1]));
    }
    constexpr int F = 4 / S;
    constexpr int D = fs_depth(KS);
    static_assert(KS % D == 0 && D <= 6, "ring depth");
    constexpr int NFB = S == 1 ? 2 : 1;                  // blocks of a pair this wave finishes
    constexpr int NV = 16 * NFB;                         // values it finishes per pair
    constexpr int kFirst = S == 1 ? 1 : 2;               // first K step that finishes values
    constexpr int kPer = (NV + (KS - kFirst) - 1) / (KS - kFirst);         // values per step
    static_assert(KS > kFirst, "too few K steps per wave");
    typedef float f32x4 __attribute__((ext_vector_type(4)));
    extern __shared__ __attribute__((aligned(16))) u32x4 smem[];
    const int tid = threadIdx.x;
    const int lane = tid & 63, half = lane >> 5, l32 = lane & 31;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    // (S = 1: sk is 0 at compile time, which keeps the argument-table
    // index below constant; a runtime index the compiler cannot resolve
    // makes it copy the kernel arguments to scratch memory)
    const int fblk = wave % F, sk = S == 1 ? 0 : wave / F;
    const int m0 = blockIdx.x * p.fs_pixels;
    const int m_end = min(m0 + p.fs_pixels, p.m);
    const int nb = (m_end - m0 + 31) >> 5;
    const int f0 = (blockIdx.y * F + fblk) * 32;         // this wave's first filter
    const bool fvalid = f0 < p.coutp;
    const int co = f0 + l32;
    const bool co_ok = co < p.cout;
    const int cwh = p.cwe >> 1;
    const int ksteps = p.kh * p.kw * cwh;
    const int TR = p.tile_rows, PW = p.pw, plane = TR * PW;
    u32x4 *atile = smem;                                 // [cwe][TR][PW] e2m1
    // past the A tile: the exchange buffer (S > 1)
    f32x4 *red = reinterpret_cast<f32x4 *>(smem + p.cwe * plane);

    const MfmaParams g = pinned_geometry(p);     // (geometry in scalar registers)
    int row0, col0;
    mfma_pixel(g, m0, row0, col0);
    // the region's first padded column
    const int wc0 = WIN ? col0 : 0;
    // the region's first chunk (its loads before the filters': the widening
    // needs it first)
    std::conditional_t<QF, RegionChunkF, RegionChunk> rch;
    if constexpr (QF)
        region_load_f<kMfmaThreads>(g, row0, wc0, plane, tid, 0, rch);
    else
        region_load<kMfmaThreads>(g, row0, wc0, plane, tid, 0, rch);

    // ---- per-lane output-transform parameters of filter co, as buffer
    // loads issued between the region's and the filters' (so that waiting
    // for them leaves the filters in flight), used once the region is
    // widened (an
    // absent array is an empty buffer: its loads read zeros, replaced by the
    // default).  A flipped filter (bitpacked output) is computed negated:
    // its widened weights get their sign bits inverted, so the accumulator
    // holds -dot, and the bit dot >= T becomes -dot < 1 - T (integers;
    // +-infinity stay exact), the same compare as for every other filter.
    float ep_a = 0.0f, ep_b = 0.0f;
    uint32_t flip_word = 0;
    {
        const int cc4 = min(co, p.cout - 1) * 4;
        const uint32_t cb = (uint32_t)p.cout * 4u;
        if constexpr (OUT == OUT_BITS) {
            ep_a = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(buffer_of(p.thr, cb), cc4, 0, 0));
            flip_word = __builtin_amdgcn_raw_buffer_load_b32(
                buffer_of(p.flip, p.flip ? (uint32_t)p.cwo * 4u : 0u), (f0 >> 5) * 4, 0, 0);
        } else if constexpr (OUT == OUT_FLOAT) {
            const float m = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
                buffer_of(p.mult, p.mult ? cb : 0u), cc4, 0, 0));
            const float b = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
                buffer_of(p.bias, p.bias ? cb : 0u), cc4, 0, 0));
            ep_a = p.mult ? m : 1.0f;
            ep_b = p.bias ? b : 0.0f;
        }
    }

    // ---- this wave's filters: step i is K step s = sk*KS + i = (tap t =
    // s / (Cw'/2), word pair q = s % (Cw'/2)): word 2q + half of tap t of
    // filter co, which is row 2s + half of the widened filters; and the
    // offset of the same word and tap in the A tile (lane-dependent, so it
    // stays in a VGPR).  The loads are unconditional (filters past C_out'
    // read the last one and are never stored; steps past the last read the
    // last row and are zeroed on arrival); each is a wave-uniform row
    // address plus a 32-bit lane offset.  Nothing waits for them here: the
    // first pair's K step i waits for its own (memory counters retire in
    // order), so the first products start while later filters still arrive.
    // PK: every channel of every word is valid, and the packed words are
    // loaded instead (a quarter of the bytes) and widened on arrival.
    static_assert(S * KS <= kFsMaxSteps, "offset table");
    u32x4 breg[KS];
    uint32_t bpk[PK ? KS : 1];
    int aoff[KS];
    {
        const __amdgpu_buffer_rsrc_t wb = filter_buffer(p, PK);
        constexpr int kEl = PK ? 4 : 16;                 // bytes per filter element
        const int col = (half * p.coutp + min(co, p.coutp - 1)) * kEl;
        const int hp = half * plane;
#pragma unroll
        for (int i = 0; i < KS; ++i) {
            const int row = 2 * min(sk * KS + i, ksteps - 1) * p.coutp * kEl;   // uniform
            if constexpr (PK)
                bpk[i] = __builtin_amdgcn_raw_buffer_load_b32(wb, col, row, 0);
            else
                breg[i] = __builtin_amdgcn_raw_buffer_load_b128(wb, col, row, 0);
            aoff[i] = (p.fs_koff[sk * KS + i] & 0xFFFFFF) + hp;   // (word 2q + half)
        }
    }

    // bitpacked output: the bounds of the workgroup's F filter blocks go to
    // LDS after the exchange area (one copy per filter block); after them,
    // the A-tile offset of every pixel's window origin (the pixel blocks'
    // bases in the loop: one LDS read each instead of the divisions of
    // mfma_pixel), computed while the region's loads are in flight
    float *thrs = reinterpret_cast<float *>(smem + p.cwe * plane) + p.fs_thr_off;
    int *btab = reinterpret_cast<int *>(thrs + F * 32);
    for (int t = tid; t < nb * 32; t += kMfmaThreads) {
        int prow, pcol;
        mfma_pixel(g, min(m0 + t, m_end - 1), prow, pcol);
        btab[t] = (prow - row0) * PW + (pcol - wc0);
    }

    // The region, widened as its words arrive (the compiler waits for them
    // here, with the filter loads still outstanding), the rest of it if any,
    // and the words past Cw.
    if constexpr (QF) {
        region_widen_f<kMfmaThreads>(g, rch, atile, plane, tid, 0);
        region_finish_f<kMfmaThreads>(g, atile, row0, wc0, plane, tid);
    } else {
        region_widen<kMfmaThreads>(g, rch, atile, plane, tid, 0);
        region_finish<kMfmaThreads>(g, atile, row0, wc0, plane, tid);
    }
    int z;
    const bool flipped = OUT == OUT_BITS && fvalid && co_ok && ((flip_word >> l32) & 1u);
    // sign bits of a flipped filter (in the widened or the packed form),
    // applied to each step's filters as they arrive (first pair)
    const uint32_t neg = OUT == OUT_BITS && flipped ? (PK ? ~0u : kFp4SignBits) : 0u;
    if constexpr (OUT == OUT_BITS) {
        ep_a = co_ok ? thr_to_dot_bound_f(ep_a, p.lo, p.hi) : -INFINITY;
        if (flipped) ep_a = 1.0f - ep_a;
        if (sk == 0 && half == 0) thrs[fblk * 32 + l32] = ep_a;
    }
    z = lds_barrier();                                   // the A tile is complete

    // Bitpacked output: the products are transposed (filters as the row
    // operand, pixels as the column operand: lane = pixel of the block, value
    // v = filter (v/4)*8 + half*4 + v%4), and each accumulator a wave
    // finishes starts at -bound instead of 0, so that the finished value is
    // dot - bound and the output bit its sign: one ALU operation per bit and
    // no lane writes.  With S > 1 only the wave that finishes a block starts
    // it at -bound (S = 1: both blocks of a pair start from one copy).
    constexpr int NT = S == 1 ? 1 : 2;
    mfma_v16f tinit[NT];
    if constexpr (OUT == OUT_BITS) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float4 t =
                reinterpret_cast<const float4 *>(thrs)[(fblk * 32 + q * 8 + half * 4 + z) >> 2];
            const float tv[4] = {t.x, t.y, t.z, t.w};
#pragma unroll
            for (int e = 0; e < 4; ++e)
#pragma unroll
                for (int b = 0; b < NT; ++b)
                    tinit[b][4 * q + e] = S == 1 || b == sk ? -tv[e] : 0.0f;
        }
    }

    // A-tile offset of the window origin of pixel block b's 32 pixels
    auto block_base = [&](int b) __attribute__((always_inline)) {
        return btab[b * 32 + l32 + z];
    };

    // ---- finishing a pair (or the last single block).  S = 1: this wave
    // finishes both blocks, from two accumulator sets that alternate by
    // pair: while a pair's products run on one set, the previous pair's
    // values are read from the other in pieces between them, so no product
    // waits for the finishing and no finishing waits for a product.  S > 1:
    // one set; wave sk < 2 finishes block sk of the pair after the other S-1
    // waves of its filter block hand it their partial sums through LDS
    // (red[(((buf*F + fblk)*2 + block)*(S-1) + slot)*4 + quad] rows of 64
    // lanes, slot = the writer's rank among the other waves, two alternating
    // buffers); waves sk >= 2 finish nothing.  The values leave the
    // accumulators (into fin, or into LDS for another wave) before the next
    // pair's first products overwrite them.
    // (accumulator blocks and sets are picked with constant indices only: a
    // runtime index would move them to scratch memory)
    constexpr int NSET = S == 1 ? 2 : 1;
    mfma_v16f acc[NSET][2];
    // (S > 1: zero-initialized, since a wave with no block of its own in a
    // pass computes values it never stores, and reading an unassigned fin
    // there would be undefined: the compiler then may, and did, rewrite the
    // other waves' path wrongly)
    float fin[S == 1 ? 1 : NFB][16] = {};
    uint32_t word[NFB];
    int fin_b0 = 0, fin_nbp = 2;
    int buf = 0;
    auto collect_prev = [&](int nbp) __attribute__((always_inline)) {
        fin_nbp = nbp;
        if constexpr (S > 1) {
            auto move = [&](auto jc) __attribute__((always_inline)) {
                constexpr int J = decltype(jc)::value;
                if (J >= nbp) return;
                if (J == sk) {
#pragma unroll
                    for (int v = 0; v < 16; ++v) fin[0][v] = acc[0][J][v];
                } else {
                    const int slot = sk - (sk > J ? 1 : 0);
#pragma unroll
                    for (int vq = 0; vq < 4; ++vq)
                        red[((((buf * F + fblk) * 2 + J) * (S - 1) + slot) * 4 + vq) * 64 + lane + z] =
                            f32x4{acc[0][J][4 * vq], acc[0][J][4 * vq + 1], acc[0][J][4 * vq + 2],
                                  acc[0][J][4 * vq + 3]};
                }
            };
            move(std::integral_constant<int, 0>{});
            move(std::integral_constant<int, 1>{});
        }
    };
    // (S > 1) the other waves' partial sums of this wave's block
    auto collect_partner = [&]() __attribute__((always_inline)) {
        if constexpr (S > 1) {
            z = lds_barrier();
            if (sk < fin_nbp) {
#pragma unroll
                for (int slot = 0; slot < S - 1; ++slot)
#pragma unroll
                    for (int vq = 0; vq < 4; ++vq) {
                        const f32x4 r =
                            red[((((buf * F + fblk) * 2 + sk) * (S - 1) + slot) * 4 + vq) * 64 +
                                lane + z];
#pragma unroll
                        for (int e = 0; e < 4; ++e) fin[0][4 * vq + e] += r[e];
                    }
            }
            buf ^= 1;
        }
    };
    // value V of block J of those this wave finishes, from accumulator set
    // PS (S = 1) or from fin (S > 1)
    auto value = [&](auto jc, auto vc, auto psc) __attribute__((always_inline)) -> float {
        constexpr int J = decltype(jc)::value, V = decltype(vc)::value;
        if constexpr (S == 1)
            return acc[decltype(psc)::value][J][V];
        else
            return fin[J][V];
    };
    // value N of the finishing order: block N/16 of those this wave
    // finishes, value N%16; a block's output is stored after its last value.
    // No branch: values of a missing block (single last block) or of
    // filters past C_out' are computed and not stored.
    auto finish_cmp = [&](auto nc, auto psc) __attribute__((always_inline)) {
        constexpr int N = decltype(nc)::value;
        constexpr int j = N / 16, v = N % 16;
        using JC = std::integral_constant<int, j>;
        if constexpr (OUT == OUT_BITS) {
            // the bit of a value (dot - bound) is its sign.  The values are
            // taken last to first (value vv = 15 - v at step v), each sign
            // shifted into the word from the right (one v_alignbit_b32), so
            // that bit vv of the word ends as value vv's sign.  Value vv is
            // filter (vv/4)*8 + half*4 + vv%4: after the last one, nibble q
            // of the word moves to nibble 2q + half, and the two halves of
            // the pixel (lanes l and l + 32) are merged.  Then lane < 32
            // stores block 0's word of pixel lane, lane >= 32 block 1's
            // (S = 1); with S > 1 lanes < 32 store the wave's block.
            constexpr int vv = 15 - v;
            const uint32_t u = __float_as_uint(value(JC{}, std::integral_constant<int, vv>{}, psc));
            uint32_t w = v == 0 ? u >> 31 : __builtin_amdgcn_alignbit(word[j], u, 31);
            if constexpr (v == 15) {
                w = (w | (w << 8)) & 0x00FF00FFu;
                w = ((w | (w << 4)) & 0x0F0F0F0Fu) << (4 * half);
                const auto sw = __builtin_amdgcn_permlane32_swap(w, w, false, false);
                w = sw[0] | sw[1];
            }
            word[j] = w;
            if constexpr (v == 15 && j == NFB - 1) {
                const int blk = S == 1 ? half : sk;      // block of the pair
                const uint32_t out_word = NFB == 2 && half ? word[NFB - 1] : word[0];
                const int m = m0 + (fin_b0 + blk) * 32 + l32;
                if (fvalid && blk < fin_nbp && (S == 1 || lane < 32) && m < m_end)
                    reinterpret_cast<uint32_t *>(p.out)[(size_t)m * p.cwo + (f0 >> 5)] = out_word;
            }
        } else {
            const int blk = S == 1 ? j : sk;             // block of the pair
            const bool store = fvalid && blk < fin_nbp;
            const int mw = m0 + (fin_b0 + blk) * 32;
            const int m = mw + (v >> 2) * 8 + half * 4 + (v & 3);
            const int c = min(max((int)value(JC{}, std::integral_constant<int, v>{}, psc), p.lo),
                              p.hi);
            if (store && co_ok && m < m_end) {
                if constexpr (OUT == OUT_FLOAT)
                    reinterpret_cast<float *>(p.out)[(size_t)m * p.cout + co] =
                        __builtin_fmaf((float)c, ep_a, ep_b);
                else
                    reinterpret_cast<int32_t *>(p.out)[(size_t)m * p.cout + co] = c;
            }
        }
    };
    // values [LO, HI) of the finishing order, from set PS
    auto finish_range = [&](auto psc, auto loc, auto hic) __attribute__((always_inline)) {
        constexpr int LO = decltype(loc)::value, HI = decltype(hic)::value;
        if constexpr (LO < HI)
            for_each_index([&](auto uc) __attribute__((always_inline)) {
                finish_cmp(std::integral_constant<int, LO + decltype(uc)::value>{}, psc);
            }, std::make_integer_sequence<int, HI - LO>{});
    };
    // finish the blocks in accumulator set PS at once (outside the pipeline)
    auto finish_all = [&](int nbp, auto psc) __attribute__((always_inline)) {
        collect_prev(nbp);
        collect_partner();
        finish_range(psc, std::integral_constant<int, 0>{}, std::integral_constant<int, NV>{});
    };

    // ---- the pipelined loop over pairs (and a last single block)
    const int npairs = nb >> 1;
    int base[2] = {block_base(0), block_base(min(1, nb - 1))};
    u32x4 ring[D][2];
#pragma unroll
    for (int i = 0; i < D - 1; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) ring[i][j] = atile[base[j] + aoff[i] + z];

    const mfma_v16f zero16 = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f,
                              0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
    // the widening's sign-bit mask in a VGPR (see widen_word_vm)
    uint32_t vmask;
    asm volatile("v_mov_b32 %0, 0x88888888" : "=v"(vmask));

    // NBP (2 or 1) blocks from b0 on accumulator set SET: K step i issues
    // its products with a piece of the previous pair's finishing (from the
    // other set, S = 1) after the first (the matrix pipe runs one product
    // while the wave issues the piece), then refills its ring slot with step
    // i + D (of these blocks, or of the next ones)
    auto body = [&](auto nbp_c, auto prev_c, auto set_c, int b0) __attribute__((always_inline)) {
        constexpr int NBP = decltype(nbp_c)::value;
        constexpr bool has_prev = decltype(prev_c)::value;   // a compile-time branch per step
        constexpr int SET = decltype(set_c)::value;
        constexpr auto ps_c = std::integral_constant<int, (SET + 1) % NSET>{};
        const int nxt = b0 + 2 < nb ? b0 + 2 : b0;
        int next_base[2] = {base[0], base[1]};
        if constexpr (NBP == 2) {
            next_base[0] = block_base(nxt);
            next_base[1] = block_base(min(nxt + 1, nb - 1));
        }
        if constexpr (has_prev) collect_prev(2);         // before the products overwrite them
        auto step = [&](auto ic) __attribute__((always_inline)) {
            constexpr int i = decltype(ic)::value;
            // refill slot (i + D - 1) % D, the one step i-1 used
            constexpr int nxs = i + D - 1;
            if constexpr (nxs < KS) {
#pragma unroll
                for (int j = 0; j < NBP; ++j) ring[nxs % D][j] = atile[base[j] + aoff[nxs] + z];
            } else if constexpr (NBP == 2) {
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    ring[nxs % D][j] = atile[next_base[j] + aoff[nxs - KS] + z];
            }
            asm volatile("" ::: "memory");
            __builtin_amdgcn_sched_barrier(0);
            // first pair: this step's filters have landed (the compiler waits
            // for exactly this load); they take the flip, or 0.0 past the
            // last K step (PK: and are widened here)
            if constexpr (!has_prev) {
                const uint32_t keep = sk * KS + i < ksteps ? ~0u : 0u;
                if constexpr (PK)
                    breg[i] = widen_word_vm((bpk[i] ^ neg) & keep, kFp4PlusOne & keep, vmask);
                else
                    breg[i] = (breg[i] ^ u32x4{neg, neg, neg, neg}) & u32x4{keep, keep, keep, keep};
            }
            // finishing piece: values [lo, hi) after the first product
            constexpr int lo = i >= kFirst ? (i - kFirst) * kPer : NV;
            constexpr int hi = lo + kPer < NV ? lo + kPer : NV;
#pragma unroll
            for (int j = 0; j < NBP; ++j) {
                if constexpr (OUT == OUT_BITS)
                    acc[SET][j] = mfma_fp4(breg[i], ring[i % D][j],
                                           i == 0 ? tinit[j % NT] : acc[SET][j]);
                else
                    acc[SET][j] = mfma_fp4(ring[i % D][j], breg[i], i == 0 ? zero16 : acc[SET][j]);
                // pin the product here (it touches no memory and would move)
                asm volatile("" : "+a"(acc[SET][j]) : : "memory");
                if constexpr (has_prev) {
                    if (j == 0) {
                        if constexpr (S > 1 && i == 1) collect_partner();
                        finish_range(ps_c, std::integral_constant<int, lo>{},
                                     std::integral_constant<int, hi>{});
                    }
                }
                // keep each piece here: a compiler memory barrier for the
                // passes that move loads and stores, a scheduling barrier for
                // the machine scheduler
                asm volatile("" ::: "memory");
                __builtin_amdgcn_sched_barrier(0);
            }
        };
        for_each_index(step, std::make_integer_sequence<int, KS>{});
        base[0] = next_base[0];
        base[1] = next_base[1];
        fin_b0 = b0;
    };
    constexpr auto two = std::integral_constant<int, 2>{};
    constexpr auto one = std::integral_constant<int, 1>{};
    constexpr auto yes = std::integral_constant<bool, true>{};
    constexpr auto no = std::integral_constant<bool, false>{};
    constexpr auto set0 = std::integral_constant<int, 0>{};
    constexpr auto set1 = std::integral_constant<int, NSET - 1>{};
    // the last single block (nb odd) on the set after `last`, then the
    // finishing of whatever is left
    auto tail = [&](auto last_c) __attribute__((always_inline)) {
        constexpr auto nxt_c = std::integral_constant<int, (decltype(last_c)::value + 1) % NSET>{};
        if (nb & 1) {
            body(one, yes, nxt_c, nb - 1);
            finish_all(1, nxt_c);
        } else {
            finish_all(2, last_c);
        }
    };
    // (the bodies after the first are reached only through it, so that the
    // compiler's counter waits find every filter load retired there, and
    // wait for nothing, stores included, inside them)
    if (npairs > 0) {
        body(two, no, set0, 0);
        if constexpr (NSET == 1) {
            for (int pidx = 1; pidx < npairs; ++pidx) body(two, yes, set0, 2 * pidx);
            tail(set0);
        } else {
            // pairs alternate between the sets: unrolled by two so that
            // every set index is a constant
            int pidx = 1;
            for (; pidx + 1 < npairs; pidx += 2) {
                body(two, yes, set1, 2 * pidx);
                body(two, yes, set0, 2 * pidx + 2);
            }
            if (pidx < npairs) {
                body(two, yes, set1, 2 * pidx);
                tail(set1);
            } else {
                tail(set0);
            }
        }
    } else if (nb & 1) {
        body(one, no, set0, nb - 1);
        finish_all(1, set0);
    }
}

}  // namespace lce
