// Launchers of the kernels compiled in their own translation units (the
// matrix-core kernels and the quantize-fused convolution, compiled in
// parallel); the C ABI in lce.hip plans a launch and calls one of these.
// out_type takes lce_out_type values, which equal the kernels' OutKind
// values.
#pragma once

#include <hip/hip_runtime.h>

#include "bconv_mfma.hpp"

namespace lce {

// pixel-split schedule: CC channel words per chunk, NBLK filter blocks, MB
// pixel blocks per wave
void launch_mfma_pixel(const MfmaParams &p, int out_type, int cc, int nblk, int mb, dim3 grid,
                       size_t lds, hipStream_t stream);
// K-split schedule: tile of 32*MBW pixels x 32*NBLK filters; qf: float32
// input, binarized while staged
void launch_mfma_ksplit(const MfmaParams &p, int out_type, int nblk, int mbw, bool qf,
                        dim3 grid, size_t lds, hipStream_t stream);
// filter-stationary schedule: instance (KS, S);
// pk: load the packed filter copy; qf: float32 input, binarized while staged
void launch_mfma_fs(const MfmaParams &p, int ks, int s, bool pk, bool qf, int out_type,
                    dim3 grid, size_t lds, hipStream_t stream);
// the same, each workgroup staging only its share's window of padded columns
// (p.pw = the window's width; every share within one output row)
void launch_mfma_fs_window(const MfmaParams &p, int ks, int s, bool pk, bool qf, int out_type,
                           dim3 grid, size_t lds, hipStream_t stream);

// quantize-fused XOR/POPCOUNT convolution (float input, Cw = C_in/32 words
// per pixel): whether an instance exists, and its launch
bool has_quant_instance(int cw, int kh, int kw);
void launch_bconv2d_quant(const BconvParams &p, int out_type, dim3 grid, size_t lds,
                          hipStream_t stream);
}  // namespace lce
