// Launchers of the filter-stationary instances, one filter block per wave,
// for whole padded rows (WIN = false, mfma_fs.hip) or each share's window of
// columns (WIN = true, mfma_fs_win.hip): two translation units, compiled in
// parallel.
#pragma once

#include "launch.hpp"

namespace lce {
namespace fs_launch {

template <int KS, int S, bool PK, bool QF, bool WIN>
void launch_pk(const MfmaParams &p, int out, dim3 grid, size_t lds, hipStream_t st) {
    const dim3 block(kMfmaThreads);
    if (out == OUT_FLOAT)
        hipLaunchKernelGGL((bconv2d_mfma_fs_kernel<KS, S, OUT_FLOAT, PK, QF, WIN>), grid, block,
                           lds, st, p);
    else if (out == OUT_BITS)
        hipLaunchKernelGGL((bconv2d_mfma_fs_kernel<KS, S, OUT_BITS, PK, QF, WIN>), grid, block,
                           lds, st, p);
    else
        hipLaunchKernelGGL((bconv2d_mfma_fs_kernel<KS, S, OUT_INT, PK, QF, WIN>), grid, block,
                           lds, st, p);
}

template <int KS, int S, bool WIN>
void launch_shape(const MfmaParams &p, bool pk, bool qf, int out, dim3 grid, size_t lds,
                  hipStream_t st) {
    if (qf) {
        if (pk)
            launch_pk<KS, S, true, true, WIN>(p, out, grid, lds, st);
        else
            launch_pk<KS, S, false, true, WIN>(p, out, grid, lds, st);
    } else if (pk) {
        launch_pk<KS, S, true, false, WIN>(p, out, grid, lds, st);
    } else {
        launch_pk<KS, S, false, false, WIN>(p, out, grid, lds, st);
    }
}

// pk: every channel of every packed word is valid (C_in = 32*Cw'), so the
// kernel loads the packed copy of the filters and widens it itself; qf: the
// input is float32, binarized while the region is staged
template <bool WIN>
void launch(const MfmaParams &p, int ks, int s, bool pk, bool qf, int out, dim3 grid,
            size_t lds, hipStream_t st) {
    if (ks == 9 && s == 1) launch_shape<9, 1, WIN>(p, pk, qf, out, grid, lds, st);
    else if (ks == 18 && s == 1) launch_shape<18, 1, WIN>(p, pk, qf, out, grid, lds, st);
    else if (ks == 5 && s == 2) launch_shape<5, 2, WIN>(p, pk, qf, out, grid, lds, st);
    else if (ks == 9 && s == 2) launch_shape<9, 2, WIN>(p, pk, qf, out, grid, lds, st);
    else if (ks == 18 && s == 2) launch_shape<18, 2, WIN>(p, pk, qf, out, grid, lds, st);
    else launch_shape<18, 4, WIN>(p, pk, qf, out, grid, lds, st);
}

}  // namespace fs_launch
}  // namespace lce
