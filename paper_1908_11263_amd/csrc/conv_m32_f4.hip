// INT-2 and INT-1 convolution on the e2m1 (FP4) matrix instruction:
// instantiations of the 32x32 implicit-GEMM kernel in FP4 mode.
#include "conv_m32_impl.h"

namespace qnn {

hipError_t launch_conv_m32_f4(const ConvArgs &a, int wm, int wn, int al16, int nw, dim3 grid, hipStream_t s)
{
    return launch_conv_m32_bits<2, true>(a, wm, wn, al16, nw, grid, s);
}

}  // namespace qnn
