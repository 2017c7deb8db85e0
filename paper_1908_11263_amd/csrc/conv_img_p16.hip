// Whole-image convolution, 16-byte input pixels (32 channels at 4 bits, 64 at
// 2 bits).
#include "conv_img_impl.h"

namespace qnn {

hipError_t launch_conv_img_p16(const ImgArgs &a, int bits, int k, int wop, int cus, hipStream_t s)
{
#define QNN_IMG(B_, K_, W_)                              \
    if (bits == B_ && k == K_ && wop == W_)              \
        return launch_img<B_, 16, K_, W_>(a, cus, s);
    QNN_IMG(4, 3, 8) QNN_IMG(4, 3, 16) QNN_IMG(4, 3, 32)
    QNN_IMG(4, 5, 8) QNN_IMG(4, 5, 16) QNN_IMG(4, 5, 32)
    QNN_IMG(2, 3, 8) QNN_IMG(2, 3, 16) QNN_IMG(2, 3, 32)
#undef QNN_IMG
    return hipErrorInvalidValue;
}

}  // namespace qnn
