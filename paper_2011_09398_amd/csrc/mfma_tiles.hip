// Launchers of the pixel-split and K-split matrix-core schedules.
#include "launch.hpp"

namespace lce {
namespace {

template <int CC, int OUT, int MB>
void launch_mfma_mb(const MfmaParams &p, int nblk, dim3 grid, size_t lds, hipStream_t s) {
    const dim3 block(kMfmaThreads);
    if (nblk == 4)
        hipLaunchKernelGGL((bconv2d_mfma_kernel<CC, OUT, 4, MB>), grid, block, lds, s, p);
    else if (nblk == 2)
        hipLaunchKernelGGL((bconv2d_mfma_kernel<CC, OUT, 2, MB>), grid, block, lds, s, p);
    else
        hipLaunchKernelGGL((bconv2d_mfma_kernel<CC, OUT, 1, MB>), grid, block, lds, s, p);
}

template <int CC, int OUT>
void launch_mfma(const MfmaParams &p, int nblk, int mb, dim3 grid, size_t lds,
                 hipStream_t s) {
    if (mb == 2)
        launch_mfma_mb<CC, OUT, 2>(p, nblk, grid, lds, s);
    else
        launch_mfma_mb<CC, OUT, 1>(p, nblk, grid, lds, s);
}

// (tiles of at most eight 32x32 blocks: MBW = 4 takes NBLK <= 2)
template <int OUT, int MBW, bool QF>
void launch_mfma_ks_mb(const MfmaParams &p, int nblk, dim3 grid, size_t lds, hipStream_t s) {
    const dim3 block(kMfmaThreads);
    constexpr int kWide = MBW == 4 ? 2 : 4;
    if (nblk == 4)
        hipLaunchKernelGGL((bconv2d_mfma_ks_kernel<OUT, kWide, MBW, QF>), grid, block, lds, s, p);
    else if (nblk == 2)
        hipLaunchKernelGGL((bconv2d_mfma_ks_kernel<OUT, 2, MBW, QF>), grid, block, lds, s, p);
    else
        hipLaunchKernelGGL((bconv2d_mfma_ks_kernel<OUT, 1, MBW, QF>), grid, block, lds, s, p);
}

template <int OUT, bool QF>
void launch_mfma_ks(const MfmaParams &p, int nblk, int mbw, dim3 grid, size_t lds,
                    hipStream_t s) {
    if (mbw == 4)
        launch_mfma_ks_mb<OUT, 4, QF>(p, nblk, grid, lds, s);
    else if (mbw == 2)
        launch_mfma_ks_mb<OUT, 2, QF>(p, nblk, grid, lds, s);
    else
        launch_mfma_ks_mb<OUT, 1, QF>(p, nblk, grid, lds, s);
}

template <bool QF>
void launch_mfma_ks_out(const MfmaParams &p, int out_type, int nblk, int mbw, dim3 grid,
                        size_t lds, hipStream_t stream) {
    switch (out_type) {
        case OUT_FLOAT: launch_mfma_ks<OUT_FLOAT, QF>(p, nblk, mbw, grid, lds, stream); break;
        case OUT_BITS: launch_mfma_ks<OUT_BITS, QF>(p, nblk, mbw, grid, lds, stream); break;
        default: launch_mfma_ks<OUT_INT, QF>(p, nblk, mbw, grid, lds, stream); break;
    }
}

}  // namespace

void launch_mfma_pixel(const MfmaParams &p, int out_type, int cc, int nblk, int mb, dim3 grid,
                       size_t lds, hipStream_t stream) {
    switch (out_type * 2 + (cc == 4)) {
        case OUT_FLOAT * 2 + 0: launch_mfma<2, OUT_FLOAT>(p, nblk, mb, grid, lds, stream); break;
        case OUT_FLOAT * 2 + 1: launch_mfma<4, OUT_FLOAT>(p, nblk, mb, grid, lds, stream); break;
        case OUT_BITS * 2 + 0: launch_mfma<2, OUT_BITS>(p, nblk, mb, grid, lds, stream); break;
        case OUT_BITS * 2 + 1: launch_mfma<4, OUT_BITS>(p, nblk, mb, grid, lds, stream); break;
        case OUT_INT * 2 + 0: launch_mfma<2, OUT_INT>(p, nblk, mb, grid, lds, stream); break;
        default: launch_mfma<4, OUT_INT>(p, nblk, mb, grid, lds, stream); break;
    }
}

void launch_mfma_ksplit(const MfmaParams &p, int out_type, int nblk, int mbw, bool qf,
                        dim3 grid, size_t lds, hipStream_t stream) {
    if (qf)
        launch_mfma_ks_out<true>(p, out_type, nblk, mbw, grid, lds, stream);
    else
        launch_mfma_ks_out<false>(p, out_type, nblk, mbw, grid, lds, stream);
}

}  // namespace lce
