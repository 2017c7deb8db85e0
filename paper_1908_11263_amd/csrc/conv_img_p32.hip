// Whole-image convolution, 32-byte input pixels (32 channels at 8 bits, 64 at
// 4 bits).
#include "conv_img_impl.h"

namespace qnn {

hipError_t launch_conv_img_p32(const ImgArgs &a, int bits, int k, int wop, int cus, hipStream_t s)
{
#define QNN_IMG(B_, K_, W_)                              \
    if (bits == B_ && k == K_ && wop == W_)              \
        return launch_img<B_, 32, K_, W_>(a, cus, s);
    QNN_IMG(8, 3, 8) QNN_IMG(8, 3, 16) QNN_IMG(8, 3, 32)
    QNN_IMG(8, 5, 8) QNN_IMG(8, 5, 16) QNN_IMG(8, 5, 32)
    QNN_IMG(4, 3, 8) QNN_IMG(4, 3, 16) QNN_IMG(4, 3, 32)
#undef QNN_IMG
    return hipErrorInvalidValue;
}

}  // namespace qnn
