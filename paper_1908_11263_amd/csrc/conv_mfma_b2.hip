// 2-bit instantiations of the MFMA implicit-GEMM convolution.
#include "conv_mfma_impl.h"

namespace qnn {

hipError_t launch_conv_mfma_b2(const ConvArgs &a, int mr, int nc, int al16, dim3 grid, hipStream_t s)
{
    return launch_conv_mfma_bits<2>(a, mr, nc, al16, grid, s);
}

}  // namespace qnn
