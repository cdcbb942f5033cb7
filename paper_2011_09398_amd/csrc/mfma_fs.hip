// Launchers of the filter-stationary schedule with one filter block per wave.
#include "launch.hpp"

namespace lce {
namespace {

struct FsShapeArg {
    int ks, s;
};

template <int KS, int S, bool PK, bool QF>
void launch_mfma_fs_pk(const MfmaParams &p, int out, dim3 grid, size_t lds,
                       hipStream_t st) {
    const dim3 block(kMfmaThreads);
    if (out == OUT_FLOAT)
        hipLaunchKernelGGL((bconv2d_mfma_fs_kernel<KS, S, OUT_FLOAT, PK, QF>), grid, block,
                           lds, st, p);
    else if (out == OUT_BITS)
        hipLaunchKernelGGL((bconv2d_mfma_fs_kernel<KS, S, OUT_BITS, PK, QF>), grid, block,
                           lds, st, p);
    else
        hipLaunchKernelGGL((bconv2d_mfma_fs_kernel<KS, S, OUT_INT, PK, QF>), grid, block,
                           lds, st, p);
}

template <int KS, int S>
void launch_mfma_fs_shape(const MfmaParams &p, bool pk, bool qf, int out, dim3 grid,
                          size_t lds, hipStream_t st) {
    if (qf) {
        if (pk)
            launch_mfma_fs_pk<KS, S, true, true>(p, out, grid, lds, st);
        else
            launch_mfma_fs_pk<KS, S, false, true>(p, out, grid, lds, st);
    } else if (pk) {
        launch_mfma_fs_pk<KS, S, true, false>(p, out, grid, lds, st);
    } else {
        launch_mfma_fs_pk<KS, S, false, false>(p, out, grid, lds, st);
    }
}

// pk: every channel of every packed word is valid (C_in = 32*Cw'), so the
// kernel loads the packed copy of the filters and widens it itself; qf: the
// input is float32, binarized while the region is staged
void launch_fs(const MfmaParams &p, FsShapeArg sh, bool pk, bool qf, int out, dim3 grid,
               size_t lds, hipStream_t st) {
    if (sh.ks == 9 && sh.s == 1) launch_mfma_fs_shape<9, 1>(p, pk, qf, out, grid, lds, st);
    else if (sh.ks == 18 && sh.s == 1) launch_mfma_fs_shape<18, 1>(p, pk, qf, out, grid, lds, st);
    else if (sh.ks == 5 && sh.s == 2) launch_mfma_fs_shape<5, 2>(p, pk, qf, out, grid, lds, st);
    else if (sh.ks == 9 && sh.s == 2) launch_mfma_fs_shape<9, 2>(p, pk, qf, out, grid, lds, st);
    else if (sh.ks == 18 && sh.s == 2) launch_mfma_fs_shape<18, 2>(p, pk, qf, out, grid, lds, st);
    else launch_mfma_fs_shape<18, 4>(p, pk, qf, out, grid, lds, st);
}

}  // namespace

void launch_mfma_fs(const MfmaParams &p, int ks, int s, bool pk, bool qf, int out_type,
                     dim3 grid, size_t lds, hipStream_t stream) {
    launch_fs(p, FsShapeArg{ks, s}, pk, qf, out_type, grid, lds, stream);
}

}  // namespace lce
