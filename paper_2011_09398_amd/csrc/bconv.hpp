// Bitpacked binary 2-D convolution (LceBConv2d, arXiv 2011.09398 Section 3.2)
// as one fused kernel: implicit im2col -> XOR/POPCOUNT GEMM -> output transform.
//
// Work decomposition (gfx950, wave64):
//   * a workgroup (4 waves) owns 64 consecutive output pixels m = (n, oy, ox)
//     and a contiguous range of filters; lane l of every wave computes
//     pixel m0 + l;
//   * the 64 pixels' im2col rows (KH*KW*Cw words each) are staged once in LDS,
//     padded taps written as 0 words (= +1.0, one-padding);
//   * a wave works on blocks of RN = 8 consecutive filters.  Their packed
//     words are uniform across the wave, so they live in scalar registers
//     (s_load) and feed v_xor_b32 as its scalar operand; the hot loop is only
//     LDS reads plus v_xor_b32 / v_bcnt_u32_b32 (popcount + accumulate);
//   * the 4 waves split the workgroup's work either over filter blocks
//     (each wave then walks `nb` blocks, reusing the staged rows) or over
//     the K range (`ks` = 2 or 4 waves per block, partial sums reduced
//     through LDS) when there are too few pixel x filter blocks to fill the
//     chip's 1024 SIMDs evenly;
//   * the accumulator stays in VGPRs and the output transform is applied
//     before anything is written.
//
// The filter words of a wave are read in the same k order as the im2col row
// (OHWI filters: k = (ky*KW + kx)*Cw + cw), so the GEMM's k loop is one
// contiguous walk over both.
//
// Output transform, with acc = sum popcount(a XOR w) and dot = K - 2*acc:
//   int32:     c = clamp(dot, lo, hi)
//   float32:   fmaf((float)c, multiplier, bias)
//   bitpacked: bit = c < threshold, evaluated exactly.  For an integer c,
//              c < t  <=>  c < ceil(t); with the clamp this is constant when
//              ceil(t) <= lo (never) or ceil(t) > hi (always), and otherwise
//              dot < ceil(t)  <=>  acc >= floor((K - ceil(t)) / 2) + 1.
//              Each workgroup turns its thresholds into that bound once
//              (thr_to_acc_bound), so a bit costs one unsigned compare.
//              An optional per-channel flip mask then inverts chosen bits
//              (the direction of a threshold folded from a negative
//              multiplier).
//
// Zero padding (TensorFlow's padding value, Section 3.2 notes it needs a
// correction): padded taps are still staged as 0 words, so the XOR/POPCOUNT
// sum is the one-padded one, and the taps outside the image are taken out
// afterwards.  With S(co, ky, kx) = sum_ci W(co, ky, kx, ci) and the window's
// in-image taps forming the rectangle [y0, y1) x [x0, x1),
//     dot_zero = dot_one - sum_{padded taps} S = (K - Total) - 2*acc + In,
// Total = sum of S over all taps and In = sum of S over the rectangle.  The
// columns [x0, x1) form one of the KW(KW+1)/2 non-empty intervals I, so with
// the per-filter table of row prefixes over column intervals
//     T[y][I] = sum over ky < y, kx in I of S(co, ky, kx),
// In = T[y1][I] - T[y0][I]: two reads per filter.  pad_table_kernel computes
// T once per filter tensor.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <climits>
#include <type_traits>

namespace lce {

enum OutKind : int { OUT_FLOAT = 0, OUT_BITS = 1, OUT_INT = 2 };

constexpr int kPix = 64;          // output pixels per workgroup (one per lane)
constexpr int kWaves = 4;         // waves per workgroup
constexpr int kThreads = kPix * kWaves;
constexpr int kRN = 8;            // filters per block (one output byte when bitpacked)
constexpr int kKC = 8;            // k words per scalar-load chunk
constexpr int kMaxNB = 4;         // filter blocks per wave
constexpr int kMaxFiltersWG = kWaves * kMaxNB * kRN;   // 128
constexpr int kSlabWords = 160;   // generic kernel: im2col words staged per pass
constexpr int kNever = INT32_MAX;   // zero-padding bound that no accumulator reaches
constexpr int kAlways = INT32_MIN;  // zero-padding bound that every accumulator reaches

// Unsigned division n / d for n < 2^31 by multiply-high (Granlund-Montgomery
// round-up variant): q = (mulhi(n, magic) + n) >> shift.
struct FastDiv {
    uint32_t d, magic, shift;
};

__host__ inline FastDiv make_fastdiv(uint32_t d) {
    uint32_t l = 0;
    while ((1ull << l) < d) ++l;                       // l = ceil(log2 d)
    const uint64_t magic = ((1ull << 32) * ((1ull << l) - d)) / d + 1;
    return FastDiv{d, (uint32_t)magic, l};
}

__device__ __forceinline__ uint32_t fast_div(uint32_t n, const FastDiv &f) {
    return (__umulhi(n, f.magic) + n) >> f.shift;
}

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
    FastDiv div_ohw;        // m -> image
    FastDiv div_ow;         // pixel within image -> row
    int32_t nb;             // filter blocks per wave (ks == 1)
    int32_t ks;             // waves sharing one block's K range (1, 2 or 4)
    int32_t fwg;            // filters per workgroup = (4 / ks) * nb * RN
    int32_t ksplit;         // K words per split (multiple of 4), ks > 1
    int32_t out_vec4;       // out is 16-byte aligned (float output may use float4 stores)
    int32_t tiles;          // static kernel: grid size when the tiles are renumbered
                            // filter-major per XCD, 0 = launch order
    FastDiv div_tile;       // static kernel, filter-major: tile index -> filter group (by grid x)
    const uint32_t *flip;   // [Cwo] or null: output bits to invert (bitpacked output)
    // (the fields above fill the first three 64-byte lines, which the static
    // kernel fetches at once; those below serve zero padding, the generic and
    // the quantize-fused kernels)
    const int32_t *padc;    // zero padding: table T [(KH+1)*KW*(KW+1)/2][Cout]
    FastDiv div_fwg;        // static kernel, zero padding: flat table index -> row
    int32_t slab;           // generic kernel: words staged per pass
    int32_t rs;             // generic kernel: LDS row stride (words)
    const float *xf;        // quantize-fused kernel: float32 input [N][H][W][32*Cw]
    int32_t band_rows;      // quantize-fused kernel: rows of the tallest input band
    int32_t band_pack;      // quantize-fused kernel: LDS word offset of the packed band
};

// LDS row stride for a row of `words` words: a multiple of 4 (16-byte rows
// for ds_read_b128) with an odd number of 16-byte quads, so the rows of
// neighbouring lanes start in different bank groups.
__host__ __device__ constexpr int row_stride(int words) {
    return ((words + 3) / 4) % 2 == 1 ? (words + 3) / 4 * 4 : (words + 3) / 4 * 4 + 4;
}

// Number of non-empty column intervals [x0, x1) of a KW-wide window, and the
// index of one of them (intervals ordered by x0, then x1).
__host__ __device__ inline int interval_count(int kw) { return kw * (kw + 1) / 2; }

__host__ __device__ inline int interval_index(int x0, int x1, int kw) {
    // intervals starting before x0: sum_{j < x0} (kw - j) = x0 * (2kw - x0 + 1) / 2
    // (unsigned: below 2^32 whenever the table fits 2^31 elements)
    return (int)((uint32_t)x0 * (uint32_t)(2 * kw - x0 + 1) / 2u) + (x1 - x0 - 1);
}

// Read-only tensors (packed filters) are read through the constant address
// space: the kernel never writes them, so a wave-uniform read there is always
// a scalar load (s_load), even after the epilogue has stored output.
typedef const __attribute__((address_space(4))) uint32_t *const_u32_ptr;

typedef const __attribute__((address_space(4))) float *const_f32_ptr;

__device__ __forceinline__ const_u32_ptr as_const(const uint32_t *p) {
    return (const_u32_ptr)p;
}

__device__ __forceinline__ const_f32_ptr as_const(const float *p) {
    return (const_f32_ptr)p;
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

// acc += popcount(x) as one v_bcnt_u32_b32 (popcount plus accumulate).
// The empty asm pins the running sum to a register after every step, so the
// compiler cannot re-associate a chunk's popcounts into an add tree (which
// costs an extra v_add3 per two words).
__device__ __forceinline__ void bcnt_acc(uint32_t &acc, uint32_t x) {
    acc = __builtin_popcount(x) + acc;
    asm("" : "+v"(acc));
}

// acc[f] += sum_k popcount(a_k XOR w[f][k]) over `nwords` words starting at
// word 0 of `arow` (LDS, 16-byte aligned) and of each filter row
// `wrow + f*kwords` (global, wave-uniform).  FULL: all RN filters exist;
// otherwise filters past `nvalid` re-read the last valid row (results
// unused) so no load leaves the tensor.
template <int RN, int KC, bool FULL>
__device__ __forceinline__ void xor_popcount(uint32_t (&acc)[RN], const uint32_t *arow,
                                             const_u32_ptr wrow, int kwords, int nwords,
                                             int nvalid) {
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
    if (k + 4 <= nwords) {
        uint32_t a[4];
        lds_read<4>(a, arow + k);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
#pragma unroll
            for (int f = 0; f < RN; ++f) {
                const int fo = FULL ? f : min(f, nvalid - 1);
                bcnt_acc(acc[f], a[j] ^ wrow[(size_t)fo * kwords + k + j]);
            }
        }
        k += 4;
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

// The bound b such that the output bit of a filter is (acc >= b); see the
// header comment.  0 = always 1, 0xFFFFFFFF = always 0 (acc < 2^31).
__device__ inline uint32_t thr_to_acc_bound(float thr, int k, int lo, int hi) {
    const double t = (double)thr;
    if (t != t) return 0xFFFFFFFFu;                          // NaN: c < NaN is false
    const double tc = ceil(t);
    if (tc <= (double)lo) return 0xFFFFFFFFu;               // c >= lo >= ceil(t)
    if (tc > (double)hi) return 0u;                          // c <= hi < ceil(t)
    const int64_t T = (int64_t)tc;                           // lo < T <= hi: int32 range
    const int64_t diff = (int64_t)k - T;
    const int64_t b = (diff >= 0 ? diff / 2 : -((-diff + 1) / 2)) + 1;   // floor(diff/2)+1
    if (b <= 0) return 0u;
    if (b >= 0xFFFFFFFFll) return 0xFFFFFFFFu;
    return (uint32_t)b;
}

// Zero padding, bitpacked output: with dot_zero = kt - 2*acc + In (kt = K -
// Total) and T = ceil(thr) inside (lo, hi], the bit is
//     dot_zero < T  <=>  2*acc - In >= kt - T + 1,
// and a constant outside.  The left side lies in [-K, 3K] (K < 2^29), so
// saturating the bound to kNever / kAlways keeps the compare exact.
__device__ inline int32_t thr_to_padz_bound(float thr, int kt, int lo, int hi) {
    const double t = (double)thr;
    if (t != t) return kNever;
    const double tc = ceil(t);
    if (tc <= (double)lo) return kNever;
    if (tc > (double)hi) return kAlways;
    const int64_t b = (int64_t)kt - (int64_t)tc + 1;
    if (b >= (int64_t)kNever) return kNever;
    if (b <= (int64_t)kAlways) return kAlways;
    return (int32_t)b;
}

// Workgroup prologue: the per-filter value the epilogue needs, for filters
// [co_wg, co_wg + n), into `bound` (LDS):
//   one padding, bitpacked output:   the accumulator bound (thr_to_acc_bound);
//   zero padding, bitpacked output:  the bound on 2*acc - In (thr_to_padz_bound);
//   zero padding, other outputs:     kt = K - Total.
// Filters past cout get "never" (bitpacked) or 0.
template <int OUT, bool PADZ>
__device__ __forceinline__ void load_bounds(const BconvParams &p, int co_wg, int n,
                                            uint32_t *bound) {
    if constexpr (PADZ || OUT == OUT_BITS) {
        // Total = T[KH][interval [0, KW)]
        const size_t total_row =
            (size_t)(p.kh * interval_count(p.kw) + interval_index(0, p.kw, p.kw)) * p.cout;
        for (int t = threadIdx.x; t < n; t += kThreads) {
            const int co = co_wg + t;
            uint32_t v;
            if constexpr (!PADZ) {
                v = co < p.cout ? thr_to_acc_bound(p.thr[co], p.k, p.lo, p.hi) : 0xFFFFFFFFu;
            } else if (co < p.cout) {
                const int kt = p.k - p.padc[total_row + co];
                v = OUT == OUT_BITS ? (uint32_t)thr_to_padz_bound(p.thr[co], kt, p.lo, p.hi)
                                    : (uint32_t)kt;
            } else {
                v = OUT == OUT_BITS ? (uint32_t)kNever : 0u;
            }
            bound[t] = v;
        }
    }
}

// Zero padding: word offsets of the two table entries of one lane's window,
// whose in-image taps are rows [y0, y1) x columns [x0, x1) (table rows
// `stride` words apart): o1 = row (y1, I), o0 = row (y0, I).  Every window of
// a padded (SAME) geometry overlaps the image, so x1 > x0.  PadWin keeps
// them as they are (table in global memory); PadWin16 packs both into one
// register (LDS table, offsets below 2^16), since the window stays live
// through the whole GEMM.
struct PadWin {
    int o1, o0;
    __device__ void get(int &a, int &b) const { a = o1; b = o0; }
};

struct PadWin16 {
    uint32_t v;
    __device__ PadWin16() : v(0) {}
    __device__ explicit PadWin16(const PadWin &w) : v((uint32_t)w.o1 | (uint32_t)w.o0 << 16) {}
    __device__ void get(int &a, int &b) const { a = (int)(v & 0xFFFFu); b = (int)(v >> 16); }
};

__device__ __forceinline__ PadWin pad_window(const BconvParams &p, int iy0, int ix0, int stride) {
    const int y0 = max(0, -iy0), y1 = max(y0, min(p.kh, p.h - iy0));
    const int x0 = max(0, -ix0), x1 = max(x0 + 1, min(p.kw, p.wd - ix0));
    const int ni = interval_count(p.kw);
    const int iv = interval_index(x0, x1, p.kw);
    return PadWin{(y1 * ni + iv) * stride, (y0 * ni + iv) * stride};
}

// In = sum of S over one lane's in-image taps, for the RN filters whose table
// column starts at `sat`.  PadWin16 (static kernel): the workgroup's columns
// staged in LDS, every column of the block readable, read as 16-byte
// vectors.  PadWin (generic kernel): the table in global memory, where
// filters past `nvalid` re-read the last valid column.
template <int RN, class Win>
__device__ __forceinline__ void inside_sum(int32_t (&in)[RN], const int32_t *sat, const Win &w,
                                           int nvalid) {
    int o1, o0;
    w.get(o1, o0);
    if constexpr (std::is_same<Win, PadWin16>::value) {
        const uint32_t *t = reinterpret_cast<const uint32_t *>(sat);
        uint32_t a[RN], b[RN];
        lds_read<RN>(a, t + o1);
        lds_read<RN>(b, t + o0);
#pragma unroll
        for (int f = 0; f < RN; ++f) in[f] = (int)(a[f] - b[f]);
    } else {
#pragma unroll
        for (int f = 0; f < RN; ++f) {
            const int fo = min(f, nvalid - 1);
            in[f] = sat[o1 + fo] - sat[o0 + fo];
        }
    }
}

// Output transform of one lane's RN accumulators (Section 3.2: the fused
// activation and the per-channel multiplier/bias, or the threshold compare,
// applied to the accumulator before it is written).  `bound` is this block's
// slice of the workgroup's per-filter values (load_bounds); `sat` and `pw`
// locate the zero-padding correction (PADZ only).
template <int RN, int OUT, bool PADZ, class Win>
__device__ __forceinline__ void epilogue(const BconvParams &p, const uint32_t (&acc)[RN],
                                         int m, int co0, const uint32_t *bound,
                                         const int32_t *sat, const Win &pw) {
    const int nvalid = min(RN, p.cout - co0);   // may be <= 0 for pad-bit blocks
    int32_t in[RN];
    if constexpr (PADZ) {
        if (nvalid > 0) {
            inside_sum<RN>(in, sat, pw, nvalid);
        } else {
#pragma unroll
            for (int f = 0; f < RN; ++f) in[f] = 0;
        }
    }
    if constexpr (OUT == OUT_BITS) {
        uint32_t b[RN];
        lds_read<RN>(b, bound);                  // broadcast read, same for all lanes
        uint32_t bits = 0;
#pragma unroll
        for (int f = 0; f < RN; ++f) {
            if constexpr (PADZ)
                bits |= (uint32_t)(2 * (int)acc[f] - in[f] >= (int)b[f]) << f;
            else
                bits |= (uint32_t)(acc[f] >= b[f]) << f;
        }
        if (p.flip) {
            const uint32_t word = as_const(p.flip)[co0 >> 5];
            uint32_t fb = (word >> (co0 & 31)) & 0xFFu;
            if (nvalid < RN) fb &= nvalid > 0 ? (1u << nvalid) - 1u : 0u;
            bits ^= fb;
        }
        uint8_t *o = reinterpret_cast<uint8_t *>(p.out) + (size_t)m * p.cwo * 4 + co0 / 8;
        static_assert(RN == 8, "one output byte per filter block");
        *o = (uint8_t)bits;
    } else {
        int32_t c[RN];
        if constexpr (PADZ) {
            uint32_t kt[RN];
            lds_read<RN>(kt, bound);
#pragma unroll
            for (int f = 0; f < RN; ++f)
                c[f] = min(max((int)kt[f] - 2 * (int)acc[f] + in[f], p.lo), p.hi);
        } else {
#pragma unroll
            for (int f = 0; f < RN; ++f) c[f] = min(max(p.k - 2 * (int)acc[f], p.lo), p.hi);
        }
        if constexpr (OUT == OUT_FLOAT) {
            float *o = reinterpret_cast<float *>(p.out) + (size_t)m * p.cout + co0;
            if (nvalid == RN && p.mult && p.bias && (p.cout % 4) == 0 && p.out_vec4) {
                float y[RN];
#pragma unroll
                for (int f = 0; f < RN; ++f)
                    y[f] = __builtin_fmaf((float)c[f], as_const(p.mult)[co0 + f],
                                          as_const(p.bias)[co0 + f]);
#pragma unroll
                for (int f = 0; f < RN; f += 4)
                    *reinterpret_cast<float4 *>(o + f) =
                        make_float4(y[f], y[f + 1], y[f + 2], y[f + 3]);
            } else {
#pragma unroll
                for (int f = 0; f < RN; ++f) {
                    if (f < nvalid) {
                        const float mu = p.mult ? as_const(p.mult)[co0 + f] : 1.0f;
                        const float bi = p.bias ? as_const(p.bias)[co0 + f] : 0.0f;
                        o[f] = __builtin_fmaf((float)c[f], mu, bi);
                    }
                }
            }
        } else {
            int32_t *o = reinterpret_cast<int32_t *>(p.out) + (size_t)m * p.cout + co0;
#pragma unroll
            for (int f = 0; f < RN; ++f)
                if (f < nvalid) o[f] = c[f];
        }
    }
}

// Decompose pixel m into (image, oy, ox) and return the image's base word
// offset plus the window origin.
__device__ __forceinline__ void pixel_origin(const BconvParams &p, int m, uint32_t &img_off,
                                             int &iy0, int &ix0, int cw) {
    const uint32_t img = fast_div((uint32_t)m, p.div_ohw);
    const uint32_t r = (uint32_t)m - img * p.div_ohw.d;
    const uint32_t oy = fast_div(r, p.div_ow);
    const uint32_t ox = r - oy * (uint32_t)p.ow;
    img_off = img * (uint32_t)(p.h * p.wd * cw);
    iy0 = (int)oy * p.sh - p.pt;
    ix0 = (int)ox * p.sw - p.pl;
}

// Accumulate one filter block over [k_lo, k_hi) of the staged rows.
// co0, k_lo and k_hi are wave-uniform; readfirstlane states it, so the filter
// words are always fetched with scalar loads whatever control flow
// surrounds the call.
template <int RN, int KC>
__device__ __forceinline__ void block_gemm(uint32_t (&acc)[RN], const uint32_t *arow,
                                           const uint32_t *w, int kwords, int co0, int cout,
                                           int k_lo, int k_hi) {
#pragma unroll
    for (int f = 0; f < RN; ++f) acc[f] = 0;
    co0 = __builtin_amdgcn_readfirstlane(co0);
    k_lo = __builtin_amdgcn_readfirstlane(k_lo);
    k_hi = __builtin_amdgcn_readfirstlane(k_hi);
    if (co0 >= cout) return;
    const const_u32_ptr wrow = as_const(w) + (size_t)co0 * kwords + k_lo;
    if (co0 + RN <= cout)
        xor_popcount<RN, KC, true>(acc, arow + k_lo, wrow, kwords, k_hi - k_lo, RN);
    else
        xor_popcount<RN, KC, false>(acc, arow + k_lo, wrow, kwords, k_hi - k_lo, cout - co0);
}

// The per-workgroup schedule after staging: `nb` blocks per wave (ks == 1),
// or ks waves per block with an LDS reduction of the partial sums.
// Block fl (first filter co_wg + fl) finds its epilogue values at bound + fl
// and its correction-table column at sat + fl.
template <int RN, int KC, int OUT, bool PADZ, class Win>
__device__ __forceinline__ void compute_and_store(const BconvParams &p, const uint32_t *arow,
                                                  int kwords, int wave, int lane, int m,
                                                  int co_wg, const uint32_t *bound,
                                                  const int32_t *sat, const Win &pw,
                                                  uint32_t *red) {
    const bool px_ok = m < p.m;
    const int limit = OUT == OUT_BITS ? p.cwo * 32 : p.cout;
    if (p.ks == 1) {
        for (int b = 0; b < p.nb; ++b) {
            const int fl = (wave * p.nb + b) * RN;
            const int co0 = co_wg + fl;
            if (co0 >= limit) break;
            uint32_t acc[RN];
            block_gemm<RN, KC>(acc, arow, p.w, kwords, co0, p.cout, 0, kwords);
            if (px_ok) epilogue<RN, OUT, PADZ>(p, acc, m, co0, bound + fl, sat + fl, pw);
        }
        return;
    }
    // ks waves per block: wave = group * ks + part
    const int part = wave % p.ks;
    const int group = wave / p.ks;
    const int fl = group * RN;
    const int co0 = co_wg + fl;
    const int k_lo = min(part * p.ksplit, kwords);
    const int k_hi = min(k_lo + p.ksplit, kwords);
    uint32_t acc[RN];
    block_gemm<RN, KC>(acc, arow, p.w, kwords, co0, p.cout, k_lo, k_hi);
    __syncthreads();   // `red` aliases the staged rows: every wave is done reading them
    if (part != 0) {
#pragma unroll
        for (int f = 0; f < RN; ++f) red[(wave * RN + f) * kPix + lane] = acc[f];
    }
    __syncthreads();
    if (part == 0 && co0 < limit) {
        for (int q = 1; q < p.ks; ++q)
#pragma unroll
            for (int f = 0; f < RN; ++f) acc[f] += red[((wave + q) * RN + f) * kPix + lane];
        if (px_ok) epilogue<RN, OUT, PADZ>(p, acc, m, co0, bound + fl, sat + fl, pw);
    }
}

typedef __attribute__((address_space(1))) void global_void;
typedef __attribute__((address_space(3))) void lds_void;

// Zero padding: copy the workgroup's columns of the correction table into
// LDS, densely (`sat`: ROWS rows of p.fwg words), by LDS DMA
// (global_load_lds): one instruction moves 64 consecutive words of the flat
// index c*fwg + fl, lane l's word landing at word l of the destination, so
// no register holds them and the copies are in flight together with the
// staging loads.  Columns past cout re-read a valid column (never used), and
// the last instruction's lanes past the table write the LDS slack that
// table_lds_words() adds.
template <int ROWS>
__device__ __forceinline__ void stage_table(const BconvParams &p, int co_wg, int wave, int lane,
                                            int32_t *sat) {
    const int words = ROWS * p.fwg;
    for (int u = wave; u * 64 < words; u += kWaves) {
        const int idx = min(u * 64 + lane, words - 1);
        const int c = (int)fast_div((uint32_t)idx, p.div_fwg);
        const int co = min(co_wg + (idx - c * p.fwg), p.cout - 1);
        const int32_t *src = p.padc + (size_t)c * p.cout + co;
        __builtin_amdgcn_global_load_lds((global_void *)src, (lds_void *)(sat + u * 64), 4, 0, 0);
    }
}

// LDS words the static kernel's table needs: `rows` rows of fwg words,
// rounded up to whole 64-word DMA instructions.
__host__ inline int table_lds_words(int rows, int fwg) { return (rows * fwg + 63) / 64 * 64; }

// The LDS DMA of stage_table completes with the wave's vector-memory counter;
// waiting for it to reach 0 before the barrier makes the table visible to
// every wave of the workgroup.  (s_waitcnt vmcnt(0): expcnt and lgkmcnt
// fields at their maxima, i.e. not waited on.)
__device__ __forceinline__ void wait_table() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// VEC words of a raw buffer (gfx9 buffer resource: base, byte size, no
// stride) at byte offset `off`; an offset at or past the size reads zeros.
template <int VEC>
__device__ __forceinline__ typename VecOf<VEC>::type buffer_vec(__amdgpu_buffer_rsrc_t r, int off) {
    if constexpr (VEC == 4) {
        const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
        return uint4{v[0], v[1], v[2], v[3]};
    } else if constexpr (VEC == 2) {
        const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0);
        return uint2{v[0], v[1]};
    } else {
        return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0);
    }
}

// One lane's share of its im2col row (shape known at compile time): wave w
// holds taps w, w+4, ... of its pixel, CW words each, read as VEC-word
// vectors (the tensor aligned to 4*VEC bytes).  load() issues every load,
// as buffer loads of the input (the host keeps it below 2^31 bytes): a
// padded tap (or a lane past the last pixel) takes an offset past the
// input and reads 0 words, one padding, so nothing is predicated and
// store() writes every tap as loaded.
template <int CW, int KH, int KW, int VEC>
struct TapStage {
    static constexpr int kTaps = KH * KW;
    static constexpr int kIters = (kTaps + kWaves - 1) / kWaves;
    static constexpr int kVecs = CW / VEC;
    using Vec = typename VecOf<VEC>::type;
    Vec v[kIters][kVecs];

    // img_off: word offset of the pixel's image; (iy0, ix0): its window origin
    __device__ __forceinline__ void load(const BconvParams &p, uint32_t img_off, int wave,
                                         bool px_ok, int iy0, int ix0) {
        const __amdgpu_buffer_rsrc_t xb = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<uint32_t *>(p.x), (short)0,
            (int)((uint32_t)p.n * p.h * p.wd * CW * 4u), 0x00020000);
#pragma unroll
        for (int i = 0; i < kIters; ++i) {
            const int t = min(wave + i * kWaves, kTaps - 1);
            const int ky = t / KW, kx = t - (t / KW) * KW;
            const int iy = iy0 + ky, ix = ix0 + kx;
            const bool in = px_ok && (unsigned)iy < (unsigned)p.h && (unsigned)ix < (unsigned)p.wd;
            const int off = in ? (int)((img_off + ((uint32_t)iy * (uint32_t)p.wd + (uint32_t)ix) * CW) * 4u)
                               : (int)0x80000000u;
#pragma unroll
            for (int c = 0; c < kVecs; ++c) v[i][c] = buffer_vec<VEC>(xb, off + c * VEC * 4);
        }
    }

    // row: the lane's im2col row in LDS
    __device__ __forceinline__ void store(uint32_t *row, int wave) const {
#pragma unroll
        for (int i = 0; i < kIters; ++i) {
            const int t = wave + i * kWaves;
            if (t < kTaps) {
                Vec *dst = reinterpret_cast<Vec *>(row + t * CW);
#pragma unroll
                for (int c = 0; c < kVecs; ++c) dst[c] = v[i][c];
            }
        }
    }
};

// Workgroup tile (pixel block bx, filter group by) of this launch index.
// The 8 XCDs take the workgroups round-robin in launch order (index L to
// XCD L % 8), each with its own L2, so in launch order every XCD's blocks
// span all filter groups and every L2 fetches every filter.  Where the
// filters outweigh the input, the tiles are renumbered filter-major (the
// tiles of one filter group consecutive) and XCD x runs the contiguous
// range [x*q + min(x, r), ...) of the T = 8q + r tiles: each L2 then
// fetches an eighth of the filters.  (Pixel-major ranges cut the input's
// re-reads likewise where the input is larger, but measured no faster than
// the launch order.)
constexpr uint32_t kXcdCount = 8;

// The first three 64-byte lines of the kernel arguments (one field of
// each: every field the static kernel reads outside zero padding), fetched
// in one round trip at the top of the kernel: the compiler would otherwise
// load them in dependent batches (behind the tile-order branch and the
// pixel test), each first touch of a line a full memory latency.
__device__ __forceinline__ void fetch_arg_lines(const BconvParams &p) {
    asm volatile("" ::"s"(p.x), "s"(p.oh), "s"(p.div_ow.magic));
}

__device__ __forceinline__ void static_tile(const BconvParams &p, int &bx, int &by) {
    if (!p.tiles) {
        bx = blockIdx.x;
        by = blockIdx.y;
        return;
    }
    const uint32_t gx = p.div_tile.d, T = (uint32_t)p.tiles;
    const uint32_t L = blockIdx.y * gx + blockIdx.x;
    const uint32_t q = T / kXcdCount, r = T % kXcdCount, x = L % kXcdCount;
    const uint32_t t = x * q + min(x, r) + L / kXcdCount;
    const uint32_t fg = fast_div(t, p.div_tile);
    bx = (int)(t - fg * gx);
    by = (int)fg;
}

// Shape-specialized kernel: Cw, KH, KW known at compile time, so the whole
// im2col row fits one LDS slab and the filter-row offsets are immediates.
// VEC = words per global load when staging (needs x aligned to 4*VEC bytes).
// PADZ: zero padding with padded taps; the workgroup's columns of the
// correction table are staged in dynamic LDS next to the rows.
template <int CW, int KH, int KW, int VEC, int OUT, bool PADZ>
__global__ __launch_bounds__(kThreads) void bconv2d_static_kernel(BconvParams p) {
    constexpr int kTaps = KH * KW;
    constexpr int kWords = kTaps * CW;
    constexpr int kRS = row_stride(kWords);
    constexpr int kRed = kWaves * kRN * kPix;   // K-split partial sums, after the rows
    constexpr int kTableRows = (KH + 1) * KW * (KW + 1) / 2;
    __shared__ __attribute__((aligned(16))) uint32_t lds[kPix * kRS > kRed ? kPix * kRS : kRed];
    __shared__ __attribute__((aligned(16))) uint32_t bound[kMaxFiltersWG];
    extern __shared__ __attribute__((aligned(16))) int32_t sat[];   // PADZ: kTableRows rows

    fetch_arg_lines(p);
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    int bx, by;
    static_tile(p, bx, by);
    const int m = bx * kPix + lane;
    const bool px_ok = m < p.m;
    const int co_wg = by * p.fwg;
    uint32_t img_off = 0;
    int iy0 = 0, ix0 = 0;
    if (px_ok) pixel_origin(p, m, img_off, iy0, ix0, CW);

    // ---- stage the im2col rows: wave w copies taps w, w+4, ... of every pixel.
    // All global loads are issued before any LDS store.  The per-filter
    // epilogue values (and, for zero padding, the correction table) are
    // fetched while those loads are in flight.
    {
        TapStage<CW, KH, KW, VEC> taps;
        taps.load(p, img_off, wave, px_ok, iy0, ix0);
        if constexpr (PADZ) stage_table<kTableRows>(p, co_wg, wave, lane, sat);
        load_bounds<OUT, PADZ>(p, co_wg, p.fwg, bound);
        taps.store(lds + lane * kRS, wave);
    }
    if constexpr (PADZ) wait_table();
    __syncthreads();
    PadWin16 pw;
    if constexpr (PADZ) pw = PadWin16(pad_window(p, iy0, ix0, p.fwg));
    compute_and_store<kRN, kKC, OUT, PADZ>(p, lds + lane * kRS, kWords, wave, lane, m, co_wg,
                                           bound, sat, pw, lds);
}

// Generic kernel: any Cw/KH/KW, one filter block per wave.  The im2col row
// is staged in slabs of p.slab words (k range [k0, k0+slab)), one word per
// copy.  PADZ reads the correction table from global memory.
template <int OUT, bool PADZ>
__global__ __launch_bounds__(kThreads) void bconv2d_generic_kernel(BconvParams p) {
    constexpr int RN = kRN;
    extern __shared__ __attribute__((aligned(16))) uint32_t lds_dyn[];
    __shared__ __attribute__((aligned(16))) uint32_t bound[kWaves * kRN];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int m = blockIdx.x * kPix + lane;
    const bool px_ok = m < p.m;
    const int co_wg = blockIdx.y * kWaves * RN;
    load_bounds<OUT, PADZ>(p, co_wg, kWaves * RN, bound);
    uint32_t img_off = 0;
    int iy0 = 0, ix0 = 0;
    if (px_ok) pixel_origin(p, m, img_off, iy0, ix0, p.cw);
    const uint32_t *ximg = p.x + img_off;
    uint32_t *row = lds_dyn + lane * p.rs;

    const int co0 = co_wg + wave * RN;
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
            const uint32_t off = in ? ((uint32_t)iy * (uint32_t)p.wd + (uint32_t)ix) * p.cw + c : 0u;
            row[kk] = in ? ximg[off] : 0u;
        }
        __syncthreads();
        if (co0 < p.cout) {
            const const_u32_ptr wrow = as_const(p.w) + (size_t)co0 * p.kwords + k0;
            if (co0 + RN <= p.cout)
                xor_popcount<RN, kKC, true>(acc, row, wrow, p.kwords, nw, RN);
            else
                xor_popcount<RN, kKC, false>(acc, row, wrow, p.kwords, nw, p.cout - co0);
        }
    }
    if (!px_ok) return;
    if (OUT == OUT_BITS ? co0 >= p.cwo * 32 : co0 >= p.cout) return;
    PadWin pw{0, 0};
    if constexpr (PADZ) pw = pad_window(p, iy0, ix0, p.cout);
    epilogue<RN, OUT, PADZ>(p, acc, m, co0, bound + wave * RN, p.padc + co0, pw);
}

}  // namespace lce
