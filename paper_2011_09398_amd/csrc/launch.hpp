// Launchers of the matrix-core kernels, one translation unit per kernel
// family (compiled in parallel); the C ABI in lce.hip plans a launch and
// calls one of these.  out_type takes lce_out_type values, which equal the
// kernels' OutKind values.
#pragma once

#include <hip/hip_runtime.h>

#include "bconv_mfma.hpp"

namespace lce {

// pixel-split schedule: CC channel words per chunk, NBLK filter blocks, MB
// pixel blocks per wave
void launch_mfma_pixel(const MfmaParams &p, int out_type, int cc, int nblk, int mb, dim3 grid,
                       size_t lds, hipStream_t stream);
// K-split schedule: tile of 32*MBW pixels x 32*NBLK filters
void launch_mfma_ksplit(const MfmaParams &p, int out_type, int nblk, int mbw, dim3 grid,
                        size_t lds, hipStream_t stream);
// filter-stationary schedule: instance (KS, S);
// pk: load the packed filter copy
void launch_mfma_fs(const MfmaParams &p, int ks, int s, bool pk, int out_type, dim3 grid,
                     size_t lds, hipStream_t stream);
}  // namespace lce
