// 4-bit instantiations of the 32x32x32 MFMA implicit-GEMM convolution.
#include "conv_m32_impl.h"

namespace qnn {

hipError_t launch_conv_m32_b4(const ConvArgs &a, int wm, int wn, int al16, int nw, dim3 grid, hipStream_t s)
{
    return launch_conv_m32_bits<4>(a, wm, wn, al16, nw, grid, s);
}

}  // namespace qnn
