// The filter-stationary instances that stage each share's window of padded
// columns (shares within one output row).
#include "mfma_fs_launch.hpp"

namespace lce {

void launch_mfma_fs_window(const MfmaParams &p, int ks, int s, bool pk, bool qf, int out_type,
                           dim3 grid, size_t lds, hipStream_t stream) {
    fs_launch::launch<true>(p, ks, s, pk, qf, out_type, grid, lds, stream);
}

}  // namespace lce
