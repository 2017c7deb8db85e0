// Whole-image convolution, 32-byte input pixels (32 channels at 8 bits, 64 at
// 4 bits); images larger than one tile in bands of output rows (32-pixel-wide
// row tiles only).
#include "conv_img_impl.h"

namespace qnn {

hipError_t launch_conv_img_p32(const ImgArgs &a, int bits, int k, int wop, int cus, hipStream_t s)
{
#define QNN_IMG(B_, K_, W_)                              \
    if (bits == B_ && k == K_ && wop == W_)              \
        return launch_img<B_, 32, K_, W_>(a, cus, s);
#define QNN_BAND(B_, K_)                                 \
    if (bits == B_ && k == K_ && wop == 32)              \
        return launch_img<B_, 32, K_, 32, true>(a, cus, s);
    if (a.bands > 0) {
        QNN_BAND(8, 3) QNN_BAND(8, 5) QNN_BAND(4, 3)
        return hipErrorInvalidValue;
    }
    QNN_IMG(8, 3, 8) QNN_IMG(8, 3, 16) QNN_IMG(8, 3, 32)
    QNN_IMG(8, 5, 8) QNN_IMG(8, 5, 16) QNN_IMG(8, 5, 32)
    QNN_IMG(4, 3, 8) QNN_IMG(4, 3, 16) QNN_IMG(4, 3, 32)
#undef QNN_IMG
#undef QNN_BAND
    return hipErrorInvalidValue;
}

}  // namespace qnn
