// Whole-image convolution, one-word input pixels (a network's first layer),
// and half-word pixels (4 channels at 4 bits: 3 image channels and a zero
// channel).
#include "conv_img_impl.h"

namespace qnn {

hipError_t launch_conv_img_p4(const ImgArgs &a, int bits, int k, int cus, hipStream_t s)
{
#define QNN_IMG(B_, K_)                                  \
    if (bits == B_ && k == K_)                           \
        return launch_img<B_, 4, K_, 32>(a, cus, s);
    QNN_IMG(8, 3) QNN_IMG(8, 5) QNN_IMG(4, 3) QNN_IMG(4, 5) QNN_IMG(2, 3) QNN_IMG(2, 5)
#undef QNN_IMG
    return hipErrorInvalidValue;
}

hipError_t launch_conv_img_p2(const ImgArgs &a, int bits, int k, int cus, hipStream_t s)
{
    if (bits == 4 && k == 3)
        return launch_img<4, 2, 3, 32>(a, cus, s);
    if (bits == 4 && k == 5)
        return launch_img<4, 2, 5, 32>(a, cus, s);
    return hipErrorInvalidValue;
}

}  // namespace qnn
