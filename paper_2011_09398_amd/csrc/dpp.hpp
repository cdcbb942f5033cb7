// DPP lane shifts shared by the kernels that assemble packed words from
// the nibbles of neighbouring lanes.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lce {

// DPP control for "row_shr:n": lane i reads lane i-n of its row of 16 lanes;
// with bound_ctrl set, lanes whose source falls outside the row read 0.
template <int N>
__device__ __forceinline__ uint32_t row_shr(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x110 | N, 0xF, 0xF, true);
}

}  // namespace lce
