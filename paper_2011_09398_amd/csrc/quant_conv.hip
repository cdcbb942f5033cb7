// Launchers of the quantize-fused convolution (bconv_quant.hpp): one
// instance per packed word count, filter size and output kind of the shapes
// that the XOR/POPCOUNT static kernel also specializes.
#include "launch.hpp"
#include "bconv_quant.hpp"

namespace lce {
namespace {

template <int CW, int KH, int KW>
void launch_shape(const BconvParams &p, int out, dim3 grid, size_t lds, hipStream_t st) {
    const dim3 block(kThreads);
    if (out == OUT_FLOAT)
        hipLaunchKernelGGL((bconv2d_quant_kernel<CW, KH, KW, OUT_FLOAT>), grid, block, lds, st,
                           p);
    else if (out == OUT_BITS)
        hipLaunchKernelGGL((bconv2d_quant_kernel<CW, KH, KW, OUT_BITS>), grid, block, lds, st,
                           p);
    else
        hipLaunchKernelGGL((bconv2d_quant_kernel<CW, KH, KW, OUT_INT>), grid, block, lds, st,
                           p);
}

}  // namespace

bool has_quant_instance(int cw, int kh, int kw) {
    if (kh == 3 && kw == 3) return (cw >= 1 && cw <= 6) || cw == 8 || cw == 16;
    if (kh == 5 && kw == 5) return (cw >= 1 && cw <= 6) || cw == 8;
    return false;
}

void launch_bconv2d_quant(const BconvParams &p, int out_type, dim3 grid, size_t lds,
                          hipStream_t st) {
    if (p.kh == 3 && p.kw == 3) {
        switch (p.cw) {
            case 1: launch_shape<1, 3, 3>(p, out_type, grid, lds, st); return;
            case 2: launch_shape<2, 3, 3>(p, out_type, grid, lds, st); return;
            case 3: launch_shape<3, 3, 3>(p, out_type, grid, lds, st); return;
            case 4: launch_shape<4, 3, 3>(p, out_type, grid, lds, st); return;
            case 5: launch_shape<5, 3, 3>(p, out_type, grid, lds, st); return;
            case 6: launch_shape<6, 3, 3>(p, out_type, grid, lds, st); return;
            case 8: launch_shape<8, 3, 3>(p, out_type, grid, lds, st); return;
            case 16: launch_shape<16, 3, 3>(p, out_type, grid, lds, st); return;
            default: return;
        }
    }
    switch (p.cw) {
        case 1: launch_shape<1, 5, 5>(p, out_type, grid, lds, st); return;
        case 2: launch_shape<2, 5, 5>(p, out_type, grid, lds, st); return;
        case 3: launch_shape<3, 5, 5>(p, out_type, grid, lds, st); return;
        case 4: launch_shape<4, 5, 5>(p, out_type, grid, lds, st); return;
        case 5: launch_shape<5, 5, 5>(p, out_type, grid, lds, st); return;
        case 6: launch_shape<6, 5, 5>(p, out_type, grid, lds, st); return;
        case 8: launch_shape<8, 5, 5>(p, out_type, grid, lds, st); return;
        default: return;
    }
}

}  // namespace lce
